"""GPU parity of the verify step against the CPU oracle on small seeded shapes.

Shapes span several 16-key tiles and 64-key chunks with ragged tails: draft lengths
0..5, committed lengths 0..80, encoder lengths 1..150, vocab 1000.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2608_12703_amd import ad, synth
from paper_2608_12703_amd.configs import Config, MAX_POS
from paper_2608_12703_amd.harness import Session

import gpu_common
from gpu_common import (compare_sequence, device_session, oracle_model, oracle_state,
                        planted_blocks, step_taps, subset)

pytestmark = pytest.mark.gpu

UNIT = Config(name="unit", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
              dtype="bf16", batch=5, k=5, k_min=0, frames=150, frames_min=1, kv_max=80,
              geo_p=0.3, seed=3)


def _setup(dtype, seed=3):
    cfg = UNIT.with_(dtype=dtype, seed=seed)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    return cfg, params, wl


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("layout", [ad.AD_PADDED, ad.AD_PACKED])
def test_step_matches_oracle(dtype, layout):
    cfg, params, wl = _setup(dtype)
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, set(range(wl.batch)))
    sess = device_session(cfg, params, wl, layout=layout, packed_encoder=layout == ad.AD_PACKED,
                          poison=True)
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    taps = step_taps(sess, blocks)
    worst = 0.0
    for b in range(wl.batch):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
        worst = max(worst, compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]),
                                            gpu_taps=taps))
    print(f"[{dtype} layout={layout}] max logit error {worst:.3e}")
    gpu_common.kv_report(f"{dtype} layout={layout}")
    # planted agreement: acceptance is min(G, k) where the oracle is decisive
    assert np.all(res["accept_len"] <= wl.k)
    sess.commit()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sess.kv_len.cpu().numpy(), wl.n + res["accept_len"] + 1)


def test_layouts_are_bit_identical():
    cfg, params, wl = _setup("bf16")
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]) for b in range(wl.batch)]
    outs = []
    for layout, packed_enc in [(ad.AD_PADDED, False), (ad.AD_PACKED, True), (ad.AD_PACKED, False)]:
        sess = device_session(cfg, params, wl, layout=layout, packed_encoder=packed_enc)
        sess.step(blocks)
        r = sess.results()
        hid = np.concatenate([r["hidden"][[sess.row_of(b, i) for i in range(len(blocks[b]))]]
                              for b in range(wl.batch)])
        outs.append((r["accept_len"], r["out_tokens"], hid))
    for o in outs[1:]:
        np.testing.assert_array_equal(o[0], outs[0][0])
        np.testing.assert_array_equal(o[1], outs[0][1])
        np.testing.assert_array_equal(o[2].view(np.uint32), outs[0][2].view(np.uint32))


def test_sequence_result_does_not_depend_on_batch():
    cfg, params, wl = _setup("bf16")
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]) for b in range(wl.batch)]
    full = device_session(cfg, params, wl)
    full.step(blocks)
    rf = full.results()
    b = 3
    one = device_session(cfg, params, subset(wl, [b]), k_max=full.k_max, seq_ids=[b])
    one.step(blocks[b:b + 1])
    r1 = one.results()
    rows = [full.row_of(b, i) for i in range(len(blocks[b]))]
    np.testing.assert_array_equal(r1["hidden"][:len(rows)].view(np.uint32),
                                  rf["hidden"][rows].view(np.uint32))
    assert r1["accept_len"][0] == rf["accept_len"][b]


def test_gpu_speculative_equals_gpu_autoregressive():
    """Losslessness on the GPU itself: speculative rounds emit the AR tokens exactly."""
    cfg, params, wl = _setup("bf16", seed=5)
    B, steps = 3, 30
    wl3 = synth.make_step_workload(cfg, batch=B)
    sess = device_session(cfg, params, wl3, k_max=6)
    # AR reference: one token per round
    pend = [int(t) for t in wl3.t0]
    ys = [[] for _ in range(B)]
    for _ in range(steps):
        sess.step([[p] for p in pend], commit=True)
        r = sess.results()
        assert r["err"] == 0
        pend = [int(r["out_tokens"][b][0]) for b in range(B)]
        for b in range(B):
            ys[b].append(pend[b])
    # speculative: drafts planted from the AR tokens with geometric agreement
    sess.set_kv_len(wl3.n)
    g = np.random.default_rng(11)
    got = [[] for _ in range(B)]
    pend = [int(t) for t in wl3.t0]
    while min(len(x) for x in got) < steps:
        blocks = []
        for b in range(B):
            pos = len(got[b])
            k = max(0, min(6, steps - pos))
            y = np.array(ys[b][pos: pos + k])
            G = int(g.geometric(0.35)) - 1
            d = synth.plant_drafts(y, G, g.integers(0, cfg.vocab - 1, k), g.integers(0, cfg.vocab, k))
            blocks.append(np.concatenate([[pend[b]], d[:len(y)]]))
        sess.step(blocks, commit=True)
        r = sess.results()
        assert r["err"] == 0
        for b in range(B):
            a = int(r["accept_len"][b])
            got[b] += [int(t) for t in r["out_tokens"][b][: a + 1]]
            pend[b] = got[b][-1]
    for b in range(B):
        assert got[b][:steps] == ys[b], f"sequence {b} diverged from AR"


def test_device_detected_errors_skip_the_sequence():
    cfg, params, wl = _setup("bf16")
    sess = device_session(cfg, params, wl)
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]) for b in range(wl.batch)]
    blocks[1] = blocks[1].copy()
    blocks[1][0] = cfg.vocab + 5                       # token outside the vocabulary
    sess.step(blocks, commit=True)
    r = sess.results()
    assert r["err"] & ad.AD_ERR_TOKEN
    assert r["accept_len"][1] == -1 and np.all(r["out_tokens"][1] == -1)
    assert r["kv_len"][1] == wl.n[1]                   # not advanced
    assert np.all(r["accept_len"][[0, 2, 3, 4]] >= 0)
    # a page outside the pool
    sess.err_flag.zero_()
    sess.set_kv_len(wl.n)
    page = int(sess.block_table[2, 0].item())
    sess.block_table[2, 0] = sess.num_pages + 3
    blocks[1][0] = wl.t0[1]
    sess.step(blocks)
    r = sess.results()
    assert r["err"] & ad.AD_ERR_PAGE and r["accept_len"][2] == -1
    # a block running past the last position
    sess.err_flag.zero_()
    sess.block_table[2, 0] = page
    n = wl.n.copy()
    n[3] = MAX_POS - len(blocks[3]) + 1
    sess.set_kv_len(n)
    sess.step(blocks)
    r = sess.results()
    assert r["err"] & ad.AD_ERR_LENGTH and r["accept_len"][3] == -1


def test_block_ending_at_last_position():
    cfg, params, wl = _setup("bf16")
    model = oracle_model(cfg, params)
    b = 0
    k = int(wl.k[b])
    n = MAX_POS - 1 - k
    wl.n[b] = n
    sess = device_session(cfg, params, wl)
    blocks = [np.concatenate([[wl.t0[i]], wl.fill_any[i]]) for i in range(wl.batch)]
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    st = oracle_state(cfg, model, b, n, int(wl.T[b]), int(wl.t0[b]))
    ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
    compare_sequence(cfg, sess, res, b, blocks[b], ref, n, gpu_taps=step_taps(sess, blocks))


def test_tiled_weights_are_bit_identical():
    """ad_model_pack only changes where the GEMMs read their weights from."""
    cfg, params, wl = _setup("bf16")
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]).astype(np.int64) for b in range(wl.batch)]
    out = []
    for pack in (True, False):
        sess = device_session(cfg, params, wl, want_logits=True)
        if not pack:
            sess.model.pack(None)
        sess.step(blocks)
        out.append(sess.results())
    for key in ("accept_len", "out_tokens", "greedy", "logits", "hidden"):
        np.testing.assert_array_equal(out[0][key], out[1][key])


def test_wide_column_lm_head_matches_oracle_and_row_major_weights():
    """The LM head's 256-column workgroups (blocks of more than 8 and up to 16 row tiles
    whose vocabulary has more than 256 column tiles): 20 sequences x 8 rows = 160 rows,
    vocab 40000 (313 column tiles, an odd count: the last workgroup's second tile lies
    past the vocabulary).  Tiled and row-major weights agree bit for bit, the logits and
    greedy tokens of planted sequences match the oracle, and each sequence's first row
    is bit-equal to its row in a one-row-per-sequence step (the 4-row-tile product)."""
    cfg = UNIT.with_(vocab=40000, batch=20, k=7, k_min=7, seed=11)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    planted = {0, 7, 19}
    blocks, _ = planted_blocks(cfg, model, wl, planted)
    out = []
    for pack in (True, False):
        sess = device_session(cfg, params, wl, want_logits=True)
        if not pack:
            sess.model.pack(None)
        sess.step(blocks)
        out.append((sess, sess.results()))
    (sess, res), (_, res_rm) = out
    assert res["err"] == 0
    for key in ("accept_len", "out_tokens", "greedy", "logits", "hidden", "margin"):
        np.testing.assert_array_equal(res[key], res_rm[key], err_msg=key)
    taps = step_taps(sess, blocks)
    for b in sorted(planted):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=taps)
    # the same pending tokens as a one-row block per sequence (20 rows: 4-row tiles)
    one = device_session(cfg, params, wl, want_logits=True, k_max=0)
    one.step([np.array(blocks[b][:1], np.int64) for b in range(wl.batch)])
    r1 = one.results()
    rows = [sess.row_of(b, 0) for b in range(wl.batch)]
    np.testing.assert_array_equal(r1["logits"].view(np.uint32), res["logits"][rows].view(np.uint32))
    np.testing.assert_array_equal(r1["greedy"], res["greedy"][rows])


@pytest.mark.parametrize("batch", [80, 160])
def test_up_projection_epilogue_at_wide_and_16_row_tiles(batch):
    """FFN-up's bias + GELU epilogue in the layouts large blocks take: d_ffn 5120 (40
    column tiles) at 640 rows runs 8-row-tile workgroups (the wide layout) and at 1280
    rows 16-row-tile workgroups.  Every sequence's first row is bit-equal to its row in a
    one-row-per-sequence step (4-row tiles), and planted sequences match the oracle."""
    cfg = UNIT.with_(d_ffn=5120, batch=batch, k=7, k_min=7, seed=13)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    planted = {0, batch - 1}
    blocks, _ = planted_blocks(cfg, model, wl, planted)
    sess = device_session(cfg, params, wl, want_logits=True)
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    taps = step_taps(sess, blocks)
    for b in sorted(planted):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=taps)
    one = device_session(cfg, params, wl, want_logits=True, k_max=0)
    one.step([np.array(blocks[b][:1], np.int64) for b in range(wl.batch)])
    r1 = one.results()
    rows = [sess.row_of(b, 0) for b in range(wl.batch)]
    for key in ("logits", "hidden"):
        np.testing.assert_array_equal(r1[key].view(np.uint32), res[key][rows].view(np.uint32), err_msg=key)
    np.testing.assert_array_equal(r1["greedy"], res["greedy"][rows])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_longest_block_64_rows(dtype):
    """The largest block a sequence may verify: 64 rows (k = 63; the row masks use all 64
    bits, four 16-row query groups), next to a one-row block, with drafts planted on the
    oracle's continuation so acceptance runs deep; the last block ends at the last
    position."""
    cfg = UNIT.with_(dtype=dtype, batch=3, k=63, k_min=63, geo_p=0.02, seed=17)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    wl.n[2] = MAX_POS - 64
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, {0, 2})
    blocks[1] = blocks[1][:1]
    wl.k[1] = 0
    sess = device_session(cfg, params, wl, k_max=63)
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    taps = step_taps(sess, blocks)
    for b in range(wl.batch):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=taps)
    sess.commit()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sess.kv_len.cpu().numpy(), wl.n + res["accept_len"] + 1)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_most_encoder_frames(dtype):
    """The most encoder frames a model may declare (max_frames 2048): six 384-frame
    chunks per cross-attention workgroup (bf16), sixteen 128-key groups (float32), in the
    padded and the packed encoder layouts."""
    cfg = UNIT.with_(dtype=dtype, batch=3, frames=2048, frames_min=2000, seed=19)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    wl.T[0] = 2048
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, set(range(wl.batch)))
    for packed in (False, True):
        sess = device_session(cfg, params, wl, packed_encoder=packed, poison=True, max_frames=2048)
        sess.step(blocks)
        res = sess.results()
        assert res["err"] == 0
        taps = step_taps(sess, blocks)
        for b in range(wl.batch):
            st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
            ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
            compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=taps)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_widest_model(dtype):
    """The widest model the library takes: 64 heads, d_model 4096 (one thread per four
    columns fills a 1024-thread row kernel; 64 attention workgroups per sequence)."""
    cfg = UNIT.with_(dtype=dtype, n_layers=1, d_model=4096, n_heads=64, d_ffn=512, batch=2, k=3, k_min=0,
                     frames=96, frames_min=1, kv_max=40, seed=23)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, set(range(wl.batch)))
    sess = device_session(cfg, params, wl)
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    for b in range(wl.batch):   # one layer: its cache values take the first layer's bar
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:])
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_most_decoder_positions(dtype):
    """The most decoder positions a model may declare (max_pos 1024: eight 128-key chunks
    per self-attention workgroup), committed prefixes up to 1018 tokens, one block ending
    at the last position."""
    cfg = UNIT.with_(dtype=dtype, max_pos=1024, batch=3, k=5, k_min=0, kv_max=1018, seed=29)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    wl.n[2] = cfg.max_pos - 1 - int(wl.k[2])
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, set(range(wl.batch)))
    sess = device_session(cfg, params, wl, poison=True)
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    taps = step_taps(sess, blocks)
    for b in range(wl.batch):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        ref = od.verify(model, st, blocks[b][1:], taps=list(range(cfg.n_layers - 1)))
        compare_sequence(cfg, sess, res, b, blocks[b], ref, int(wl.n[b]), gpu_taps=taps)
    print("committed lengths", wl.n.tolist(), "blocks", [len(x) for x in blocks])
