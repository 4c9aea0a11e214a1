"""Bit-exact batch invariance and GPU-speculative == GPU-autoregressive at the large-v3
bench shapes (32 layers, d 1280, vocab 51866, 1500 frames).

The paper's losslessness (section 3, "Speculative Loop": accepting the longest prefix that
matches the target's greedy output gives exactly the target's greedy decode) holds on
the GPU only if a row's arithmetic does not depend on the block it is verified in.  The
kernels are built for that (split counts fixed by the weight shape, key chunks at
absolute positions, fixed merge orders); the launch planner still changes tile heights
and K loops with the row count, and these tests pin that none of it changes a bit:

* seven autoregressive steps of all 32 sequences (32-row blocks: LM head with 4-row
  tiles and two K steps per barrier) against one speculative step whose drafts are the
  autoregressive tokens (224-row block: LM head with 16-row tiles): every sequence must
  accept all 6 drafts, and each block row's hidden state, logits, greedy token and
  written cache bytes must equal those of the matching autoregressive step;
* the same sequence verified alone (7 rows) and inside a ragged batch of 64 padded to
  9 rows per sequence (576 rows: the projections switch to 8-row tiles).
"""
import numpy as np
import pytest
import torch

from paper_2608_12703_amd import synth
from paper_2608_12703_amd.configs import CONFIGS
from paper_2608_12703_amd.harness import Session, upload_params

pytestmark = pytest.mark.gpu

CFG = CONFIGS["large_v3_bf16"]
K = 6
PROBE = (0, 5, 17, 31)      # sequences whose cache bytes are compared


def _session(params, wl, ids, k_max):
    """A padded session over workload `wl`; slot j draws the inputs of sequence ids[j]."""
    s = Session(CFG, params, wl.batch, k_max, wl.T, want_logits=True)
    s.prefill_encoder([synth.make_encoder(CFG, ids[j], int(wl.T[j])) for j in range(wl.batch)])
    for j in range(wl.batch):
        s.import_prefix(j, synth.make_prefix_kv(CFG, ids[j], int(wl.n[j])))
    s.set_kv_len(wl.n)
    return s


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


@pytest.fixture(scope="module")
def runs():
    params = upload_params(CFG, synth.make_params(CFG))
    wl = synth.make_step_workload(CFG)
    B = wl.batch
    ids = list(range(B))
    # autoregressive: K + 1 one-row steps of every sequence, committed each time
    ar = _session(params, wl, ids, 0)
    pend = [int(t) for t in wl.t0]
    y, hid, logit, greedy = [], [], [], []
    for _ in range(K + 1):
        ar.step([np.array([p], np.int64) for p in pend], commit=True)
        r = ar.results()
        assert r["err"] == 0
        pend = [int(r["out_tokens"][b][0]) for b in range(B)]
        y.append(pend)
        rows = [ar.row_of(b, 0) for b in range(B)]
        hid.append(r["hidden"][rows].copy())
        logit.append(r["logits"][rows].copy())
        greedy.append(r["greedy"][rows].copy())
    ar_kv = {b: ar.export_prefix(b, int(wl.n[b]) + K + 1) for b in PROBE}
    del ar
    torch.cuda.empty_cache()
    y = np.array(y).T                     # [B][K + 1]: y_1 .. y_{K+1}
    blocks = [np.concatenate([[wl.t0[b]], y[b, :K]]).astype(np.int64) for b in range(B)]
    return params, wl, blocks, y, np.array(hid), np.array(logit), np.array(greedy), ar_kv


def test_speculative_step_equals_autoregressive_steps_bit_for_bit(runs):
    params, wl, blocks, y, hid, logit, greedy, ar_kv = runs
    B = wl.batch
    sp = _session(params, wl, list(range(B)), K)
    sp.step(blocks)
    r = sp.results()
    assert r["err"] == 0
    np.testing.assert_array_equal(r["accept_len"], np.full(B, K))
    np.testing.assert_array_equal(r["out_tokens"], y)
    for i in range(K + 1):
        rows = [sp.row_of(b, i) for b in range(B)]
        np.testing.assert_array_equal(r["greedy"][rows], greedy[i])
        np.testing.assert_array_equal(_bits(r["hidden"][rows]), _bits(hid[i]), err_msg=f"row {i} hidden")
        np.testing.assert_array_equal(_bits(r["logits"][rows]), _bits(logit[i]), err_msg=f"row {i} logits")
    for b in PROBE:
        n = int(wl.n[b])
        kv = sp.export_prefix(b, n + K + 1)
        np.testing.assert_array_equal(_bits(kv[:, :, n:]), _bits(ar_kv[b][:, :, n:]),
                                      err_msg=f"seq {b} cache bytes")


@pytest.mark.parametrize("b", [5, 17])   # both in PROBE
def test_sequence_alone_and_in_ragged_batch_of_64(runs, b):
    params, wl, blocks, y, hid, logit, greedy, ar_kv = runs
    n = int(wl.n[b])
    # alone: a batch of one (7 rows)
    one = synth.StepWorkload(wl.k[[b]], wl.n[[b]], wl.T[[b]], wl.t0[[b]], wl.G[[b]],
                             [wl.fill_ne[b]], [wl.fill_any[b]])
    s1 = _session(params, one, [b], K)
    s1.step([blocks[b]])
    r1 = s1.results()
    kv1 = s1.export_prefix(0, n + K + 1)
    del s1
    # inside the ragged large-v3 batch (64 sequences, k 2..8, T 200..1500), padded to 9
    # rows per sequence; slot 10 holds sequence b, the others draw fresh inputs
    rg = synth.make_step_workload(CONFIGS["ragged_large_v3"])
    slot = 10
    k = rg.k.copy(); k[slot] = K
    nn = rg.n.copy(); nn[slot] = n
    T = rg.T.copy(); T[slot] = wl.T[b]
    t0 = rg.t0.copy(); t0[slot] = wl.t0[b]
    mix = synth.StepWorkload(k, nn, T, t0, rg.G, rg.fill_ne, rg.fill_any)
    ids = [100 + j for j in range(mix.batch)]
    ids[slot] = b
    s64 = _session(params, mix, ids, int(k.max()))
    assert s64.max_rows == 64 * 9
    blk64 = [np.concatenate([[t0[j]], rg.fill_any[j]]).astype(np.int64) for j in range(mix.batch)]
    blk64[slot] = blocks[b]
    s64.step(blk64)
    r64 = s64.results()
    assert r64["err"] == 0
    kv64 = s64.export_prefix(slot, n + K + 1)
    for i in range(K + 1):
        want_h, want_l = _bits(hid[i][b]), _bits(logit[i][b])
        np.testing.assert_array_equal(_bits(r1["hidden"][i]), want_h, err_msg=f"alone: row {i} hidden")
        np.testing.assert_array_equal(_bits(r1["logits"][i]), want_l, err_msg=f"alone: row {i} logits")
        row = s64.row_of(slot, i)
        np.testing.assert_array_equal(_bits(r64["hidden"][row]), want_h, err_msg=f"64: row {i} hidden")
        np.testing.assert_array_equal(_bits(r64["logits"][row]), want_l, err_msg=f"64: row {i} logits")
    assert int(r1["accept_len"][0]) == K and int(r64["accept_len"][slot]) == K
    np.testing.assert_array_equal(r64["out_tokens"][slot][: K + 1], y[b])
    np.testing.assert_array_equal(_bits(kv1[:, :, n:]), _bits(ar_kv[b][:, :, n:]))
    np.testing.assert_array_equal(_bits(kv64[:, :, n:]), _bits(kv1[:, :, n:]))

