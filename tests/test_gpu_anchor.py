"""GPU parity of the verification-attention anchor readout against the oracle.

Paper, section "Correction and Cost", paragraph "Verification-Attention Correction";
appendix "Runtime Correction": block row a_b's cross-attention weights at one layer,
averaged over heads, peak at the next token's audio position.  Shapes: encoder lengths
1..900 (one to three 384-frame readout chunks, ragged 32-frame tails), draft lengths
0..5, committed lengths 0..80, both storage precisions and both row layouts.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2608_12703_amd import ad, synth
from paper_2608_12703_amd.configs import Config

import gpu_common
from gpu_common import compare_anchor, device_session, oracle_model, oracle_state, planted_blocks

pytestmark = pytest.mark.gpu

UNIT = Config(name="unit_anchor", n_layers=3, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
              dtype="bf16", batch=6, k=5, k_min=0, frames=900, frames_min=1, kv_max=80,
              geo_p=0.3, seed=11)


def _run(dtype, layout, layer):
    cfg = UNIT.with_(dtype=dtype)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    blocks, _ = planted_blocks(cfg, model, wl, set(range(wl.batch)))
    sess = device_session(cfg, params, wl, layout=layout, packed_encoder=layout == ad.AD_PACKED,
                          poison=True)
    sess.anchor_layer = layer
    sess.step(blocks)
    res = sess.results()
    assert res["err"] == 0
    return cfg, model, wl, blocks, sess, res


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("layout", [ad.AD_PADDED, ad.AD_PACKED])
def test_anchor_matches_oracle(dtype, layout):
    gpu_common.ANCHOR_STATS.clear()
    for layer in (0, 2):
        cfg, model, wl, blocks, sess, res = _run(dtype, layout, layer)
        print(f"[{dtype} layout={layout} layer={layer}] T = {wl.T.tolist()}")
        compared = 0
        for b in range(wl.batch):
            st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
            ref, anc = od.verify_with_anchor(model, st, blocks[b][1:], layer)
            compared += compare_anchor(cfg, res, b, ref, anc)
        assert compared >= wl.batch - 1
    worst = max(s[2] for s in gpu_common.ANCHOR_STATS)
    equal = np.mean([s[1] for s in gpu_common.ANCHOR_STATS])
    print(f"[{dtype}] worst peak error {worst:.2e} of peak; frames equal {equal:.3f}")


def test_anchor_readout_leaves_the_step_unchanged():
    outs = []
    for layer in (-1, 1):
        cfg, model, wl, blocks, sess, res = _run("bf16", ad.AD_PADDED, layer)
        rows = [sess.row_of(b, i) for b in range(wl.batch) for i in range(len(blocks[b]))]
        outs.append((res["accept_len"], res["out_tokens"], res["logits"][rows]))
        if layer < 0:
            assert np.all(sess.out_anchor.cpu().numpy() == -1)     # not written when off
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])
    np.testing.assert_array_equal(outs[0][2].view(np.uint32), outs[1][2].view(np.uint32))


def test_anchor_layouts_identical_and_skipped_sequence():
    got = []
    for layout in (ad.AD_PADDED, ad.AD_PACKED):
        _, _, wl, blocks, sess, res = _run("bf16", layout, 1)
        got.append((res["anchor"], res["anchor_peak"]))
    np.testing.assert_array_equal(got[0][0], got[1][0])
    np.testing.assert_array_equal(got[0][1].view(np.uint32), got[1][1].view(np.uint32))
    # a sequence with an out-of-vocabulary draft is skipped: no anchor
    cfg = UNIT
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]) for b in range(wl.batch)]
    blocks[2] = blocks[2].copy()
    blocks[2][-1] = cfg.vocab + 5
    sess = device_session(cfg, params, wl)
    sess.anchor_layer = 2
    sess.step(blocks)
    res = sess.results()
    assert res["err"] & 4
    assert res["accept_len"][2] == -1 and res["anchor"][2] == -1
    ok = [b for b in range(wl.batch) if b != 2]
    assert np.all(res["anchor"][ok] >= 0) and np.all(res["anchor"][ok] < wl.T[ok])
    torch.cuda.synchronize()
