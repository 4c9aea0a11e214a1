"""GPU parity at the workloads' full sizes, in the launch configuration bench.py times.

Each test builds the whole batch exactly as the benchmark does (same generators, same
Session, same layout) and checks sampled sequences against the oracle, which recomputes
them one by one in float64 from the same seeded inputs.  Drafts fed to the oracle come
from the oracle's own greedy continuation; the other sequences of the batch get uniform
drafts (batch composition does not change a sequence's result).

Workloads (sizes as in paper_2608_12703_amd/configs.py):
  small_bf16       12 layers, d 768, batch 16, k 4, committed lengths U{0..224}
  large_v3_bf16    32 layers, d 1280, batch 32, k 6, committed lengths U{0..441}
  ragged_large_v3  batch 64, T U{200..1500}, n U{0..447}, k U{2..8}; padded vs packed
  tiny_fp32        64-token greedy decode with 4 linear draft heads
  drift_stress     decode loop with drafts that drift by +-1 token after anchors
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import accept as oa
from oracle import decoder as od
from oracle.numerics import round_f32
from paper_2608_12703_amd import ad, decode, synth
from paper_2608_12703_amd.configs import CONFIGS, SOT_TOKEN
from paper_2608_12703_amd.harness import Session, upload

from gpu_common import (MARGIN_EXCLUDE, activation_error, compare_anchor, compare_sequence,
                        device_session, kv_report, layer_input_errors, oracle_state, step_taps)

pytestmark = pytest.mark.gpu


def _sampled_step(cfg, sample, layout=ad.AD_PADDED, anchor_layer=-1):
    """One verify step of the full batch; oracle-planted drafts for `sample`.  With
    anchor_layer set, the step also reads the verification-attention anchor there.  The
    residual stream entering every layer is read back (step_taps) for the cache-value
    bound."""
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = od.Model(cfg, params)
    ids = sorted(set(sample(wl)))
    blocks, states = [], {}
    for b in range(wl.batch):
        k = int(wl.k[b])
        if b in ids:
            st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
            y, _, _ = od.ar_decode(model, st, k)
            d = synth.plant_drafts(np.array(y), int(wl.G[b]), wl.fill_ne[b], wl.fill_any[b])
            states[b] = st
        else:
            d = wl.fill_any[b]
        blocks.append(np.concatenate([[wl.t0[b]], d]).astype(np.int64))
    sess = device_session(cfg, params, wl, layout=layout, packed_encoder=layout == ad.AD_PACKED)
    sess.anchor_layer = anchor_layer
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    gpu_taps = step_taps(sess, blocks)
    taps = list(range(cfg.n_layers - 1))
    for b in ids:
        if anchor_layer >= 0:
            ref, anc = od.verify_with_anchor(model, states[b], blocks[b][1:], anchor_layer, taps=taps)
        else:
            ref = od.verify(model, states[b], blocks[b][1:], taps=taps)
        rows = [sess.row_of(b, i) for i in range(len(blocks[b]))]
        eps = layer_input_errors(gpu_taps, ref.taps, rows, cfg.n_layers)
        print(f"[{cfg.name}] seq {b}: n={int(wl.n[b])} T={int(wl.T[b])} k={int(wl.k[b])} "
              f"accept gpu {int(res['accept_len'][b])} oracle {ref.accepted}; layer-input error "
              f"{' '.join(f'{e:.1e}' for e in eps[1::max(1, len(eps) // 8)])} (every "
              f"{max(1, len(eps) // 8)}th layer), final hidden {activation_error(res['hidden'][rows], ref.hidden):.1e}")
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=gpu_taps)
        if anchor_layer >= 0:
            compare_anchor(cfg, res, b, ref, anc)
    kv_report(cfg.name)
    return sess, res, blocks, wl


def test_small_bf16_sampled_sequences():
    cfg = CONFIGS["small_bf16"]
    _sampled_step(cfg, lambda wl: [int(np.argmax(wl.n)), int(np.argmin(wl.n)), 5])


def _large_v3_sample(wl):
    """Four sequences: the longest and shortest committed prefixes, the median prefix
    and the median planted acceptance min(G, k) (the first not already taken)."""
    order_n = np.argsort(wl.n, kind="stable")
    acc = np.minimum(wl.G, wl.k)
    order_a = np.argsort(acc, kind="stable")
    picked = [int(order_n[-1]), int(order_n[0])]
    for cand in (order_n[len(order_n) // 2:], order_a[len(order_a) // 2:]):
        picked.append(next(int(c) for c in cand if int(c) not in picked))
    return picked


@pytest.mark.parametrize("half", [0, 1])
def test_large_v3_bench_configuration_sampled_sequences(half):
    """Two of the four sampled sequences per test (the oracle's float64 work for each
    takes about half a minute at this shape)."""
    cfg = CONFIGS["large_v3_bf16"]
    # with the verification-attention anchor read at three quarters of the depth
    _sampled_step(cfg, lambda wl: _large_v3_sample(wl)[2 * half: 2 * half + 2],
                  anchor_layer=3 * cfg.n_layers // 4)


def test_ragged_padded_and_packed_agree_and_match_oracle():
    cfg = CONFIGS["ragged_large_v3"]
    sample = lambda wl: [int(np.argmax(wl.k * 10000 + wl.T)), int(np.argmin(wl.T))]
    sess, res, blocks, wl = _sampled_step(cfg, sample, layout=ad.AD_PADDED,
                                          anchor_layer=3 * cfg.n_layers // 4)
    # the same step in the packed row layout with packed encoder slots
    sess2 = device_session(cfg, sess.params, wl, layout=ad.AD_PACKED, packed_encoder=True)
    sess2.anchor_layer = sess.anchor_layer
    sess2.step(blocks)
    res2 = sess2.results()
    np.testing.assert_array_equal(res2["anchor"], res["anchor"])
    np.testing.assert_array_equal(res2["anchor_peak"].view(np.uint32), res["anchor_peak"].view(np.uint32))
    np.testing.assert_array_equal(res2["accept_len"], res["accept_len"])
    np.testing.assert_array_equal(res2["out_tokens"], res["out_tokens"])
    rows = [sess.row_of(b, i) for b in range(wl.batch) for i in range(int(wl.k[b]) + 1)]
    rows2 = [sess2.row_of(b, i) for b in range(wl.batch) for i in range(int(wl.k[b]) + 1)]
    np.testing.assert_array_equal(res2["greedy"][rows2], res["greedy"][rows])
    np.testing.assert_array_equal(res2["logits"][rows2], res["logits"][rows])
    np.testing.assert_array_equal(res2["hidden"][rows2], res["hidden"][rows])


def test_tiny_fp32_decode_with_draft_heads():
    cfg = CONFIGS["tiny_fp32"]
    params = synth.make_params(cfg)
    heads = synth.make_draft_heads(cfg)
    wl = synth.make_step_workload(cfg)
    T = int(wl.T[0])
    model = od.Model(cfg, params)
    cross = od.cross_kv(model, synth.make_encoder(cfg, 0, T))
    want, want_acc, rounds = od.spec_decode_heads(model, od.new_state(model, cross, SOT_TOKEN),
                                                  heads, cfg.decode_tokens)
    ar, ar_margins, _ = od.ar_decode(model, od.new_state(model, cross, SOT_TOKEN), cfg.decode_tokens)
    assert want == ar  # the oracle itself is lossless
    r0 = od.ar_step(model, od.new_state(model, cross, SOT_TOKEN))

    def head_margin(hidden_row):
        h = np.asarray(hidden_row, np.float64)
        return min(oa.top2_margin(round_f32(np.asarray(W, np.float64) @ h)) for W in heads)

    sess = Session(cfg, params, 1, cfg.draft_heads, [T])
    sess.prefill_encoder([synth.make_encoder(cfg, 0, T)])
    sess.set_kv_len([0])
    heads_dev = upload(heads, torch.float32)
    got, got_acc, got_drafts, n_rounds = decode.decode_with_heads(sess, heads_dev, [SOT_TOKEN],
                                                                  cfg.decode_tokens)
    got, got_acc, got_drafts = got[0], [int(a[0]) for a in got_acc], [d[0] for d in got_drafts]
    print(f"[tiny_fp32] {n_rounds} rounds, accepts {got_acc}")
    # tokens agree up to the first near-tie of the target (then both stay valid greedy
    # decodes of their own, slightly different, float paths)
    cut = next((i for i, m in enumerate(ar_margins) if m < MARGIN_EXCLUDE), len(ar))
    assert got[:cut] == want[:cut]
    # per-round drafts (ad_draft_heads against the oracle's heads) and acceptance agree
    # while no draft-head or target decision is a near-tie (round 0 is the
    # autoregressive round; its hidden row drafts round 1)
    assert got_acc[0] == 0 and len(got_drafts[0]) == 0
    checked = 0
    hid, ok = r0.hidden[0], r0.margins[0] >= MARGIN_EXCLUDE
    for r, ro in enumerate(rounds):
        if not ok or head_margin(hid) < MARGIN_EXCLUDE:
            break
        want_d = od.draft_heads(heads[: len(got_drafts[r + 1])], hid)
        assert list(got_drafts[r + 1]) == list(want_d), f"round {r + 1} drafts"
        assert got_acc[r + 1] == want_acc[r], f"round {r + 1} accept"
        checked += 1
        hid, ok = ro.hidden[ro.accepted], min(ro.margins) >= MARGIN_EXCLUDE
    print(f"[tiny_fp32] drafts and accept counts compared over {checked} of {len(rounds)} drafted rounds")
    assert checked >= 8


def test_drift_stress_loop_prefix_matches_oracle():
    """128 tokens of drift-stress sequence 0 against the oracle's reference, written by
    tests/golden/make_drift_stress.py from the CPU oracle alone (ten minutes of float64
    work at this shape): its greedy continuation, margins, and the accept count of every
    round with the same planted drafts.  The sequence's misalignment anchors at 34 (+1),
    76 (+1) and 110 (-1) each force a rejection and a re-anchoring."""
    cfg = CONFIGS["drift_stress"]
    with open(os.path.join(os.path.dirname(__file__), "golden", "drift_stress_seq0.json")) as fh:
        ref = json.load(fh)
    b0, n_tokens = ref["sequence"], ref["n_tokens"]
    y, margins, ref_acc, ref_toks = ref["y"], ref["margins"], ref["accepts"], ref["tokens"]
    assert len(y) == n_tokens + cfg.k + 2
    ys0 = np.array([SOT_TOKEN] + list(y), np.int64)
    plans = [synth.make_drift_plan(cfg, b) for b in range(cfg.batch)]
    params = synth.make_params(cfg)
    T = cfg.frames
    # the device loop over the whole batch (other sequences: drafts off a uniform path)
    rng = np.random.default_rng(7)
    ys = [ys0] + [np.concatenate([[SOT_TOKEN], rng.integers(0, cfg.vocab, len(ys0) - 1)])
                  for _ in range(cfg.batch - 1)]
    sess = Session(cfg, params, cfg.batch, cfg.k, [T] * cfg.batch)
    sess.prefill_encoder([synth.make_encoder(cfg, b, T) for b in range(cfg.batch)])
    sess.set_kv_len(np.zeros(cfg.batch, np.int64))
    got, acc, rounds = decode.decode_with_drift(sess, ys, [plans[b0]] + plans[1:], cfg.k, n_tokens)
    got_acc = [int(a[b0]) for a in acc]
    print(f"[drift_stress] seq {b0}: accepts gpu {got_acc} oracle {ref_acc}")
    crossed = [(int(p), int(sg)) for p, sg in zip(plans[b0].anchors, plans[b0].signs) if p < n_tokens]
    assert len(crossed) >= 3 and {sg for _, sg in crossed} == {1, -1}
    # no oracle near-tie in the compared span (smallest margin 1.11e-3, at position 124)
    cut = next((i for i, m in enumerate(margins) if m < MARGIN_EXCLUDE), len(y))
    assert cut >= n_tokens + cfg.k + 2, f"oracle near-tie at position {cut}"
    assert got[b0][:n_tokens] == ref_toks[:n_tokens]
    # every round's accept count, including the rejection each anchor forces
    assert got_acc[: len(ref_acc)] == ref_acc
    assert sum(1 for a in ref_acc if a < cfg.k) >= len(crossed)
