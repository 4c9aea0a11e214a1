"""Pins for the oracle's verification-attention anchor readout (CPU only).

Paper, section "Correction and Cost", paragraph "Verification-Attention Correction", and
appendix "Runtime Correction": the target's audio (cross-)attention at a selected decoder
layer, averaged over heads, peaks at the audio position of the next token.

* Library: torch's ``nn.MultiheadAttention`` returns the head-averaged attention weights
  itself (``average_attn_weights=True``); a float64 torch decoder run layer by layer up
  to the probed layer must give the oracle's averaged weights and peak frame.
* Closed forms: constructed keys whose per-head weights are known exactly; equal keys
  (uniform weights, lowest-index tie-break); a single frame.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2608_12703_amd import synth


def _torch_layer(cfg, params, layer):
    t = lambda name: torch.from_numpy(np.asarray(params[name], np.float64))
    p = lambda n: t(f"l{layer}.{n}")
    mod = torch.nn.TransformerDecoderLayer(cfg.d_model, cfg.n_heads, cfg.d_ffn, dropout=0.0,
                                           activation="gelu", batch_first=True, norm_first=True,
                                           dtype=torch.float64)
    with torch.no_grad():
        mod.self_attn.in_proj_weight.copy_(p("w_qkv"))
        mod.self_attn.in_proj_bias.copy_(p("b_qkv"))
        mod.self_attn.out_proj.weight.copy_(p("w_o"))
        mod.self_attn.out_proj.bias.copy_(p("b_o"))
        mod.multihead_attn.in_proj_weight.copy_(torch.cat([p("w_xq"), p("w_xkv")]))
        mod.multihead_attn.in_proj_bias.copy_(torch.cat([p("b_xq"), p("b_xkv")]))
        mod.multihead_attn.out_proj.weight.copy_(p("w_xo"))
        mod.multihead_attn.out_proj.bias.copy_(p("b_xo"))
        mod.linear1.weight.copy_(p("w_1")); mod.linear1.bias.copy_(p("b_1"))
        mod.linear2.weight.copy_(p("w_2")); mod.linear2.bias.copy_(p("b_2"))
        for i in (1, 2, 3):
            getattr(mod, f"norm{i}").weight.copy_(p(f"ln{i}_g"))
            getattr(mod, f"norm{i}").bias.copy_(p(f"ln{i}_b"))
    return mod.eval()


def _torch_mean_xattn(cfg, params, enc, tokens, probe):
    """Head-averaged cross-attention weights [len(tokens), T] at layer ``probe``."""
    t = lambda name: torch.from_numpy(np.asarray(params[name], np.float64))
    n = len(tokens)
    x = (t("tok_emb")[torch.tensor(tokens)] + t("pos_emb")[:n])[None]
    mem = torch.from_numpy(np.asarray(enc, np.float64))[None]
    causal = torch.nn.Transformer.generate_square_subsequent_mask(n, dtype=torch.float64)
    with torch.no_grad():
        for layer in range(probe + 1):
            mod = _torch_layer(cfg, params, layer)
            if layer < probe:
                x = mod(x, mem, tgt_mask=causal, tgt_is_causal=True)
                continue
            h = mod.norm1(x)
            x = x + mod.self_attn(h, h, h, attn_mask=causal, need_weights=False)[0]
            _, w = mod.multihead_attn(mod.norm2(x), mem, mem, need_weights=True,
                                      average_attn_weights=True)
    return w[0].numpy()


@pytest.fixture(scope="module")
def tiny(tiny_cfg):
    cfg = tiny_cfg.with_(vocab=97, n_layers=3, n_heads=2)
    return cfg, synth.make_params(cfg), synth.make_encoder(cfg, 0, 41)


@pytest.mark.parametrize("probe", [0, 2])
def test_head_averaged_weights_match_torch_multihead_attention(tiny, probe):
    cfg, params, enc = tiny
    model = od.Model(cfg, params, kv_dtype="f64")
    tokens = [5, 17, 3, 3, 96, 0, 41]
    ref = _torch_mean_xattn(cfg, params, enc, tokens, probe)
    out = od.forward_block(model, od.new_state(model, od.cross_kv(model, enc), tokens[0]), tokens,
                           probe_layer=probe)
    assert out.xattn.shape == (len(tokens), cfg.n_heads, 41)
    np.testing.assert_allclose(out.xattn.mean(axis=1), ref, rtol=0, atol=1e-13)
    np.testing.assert_allclose(out.xattn.sum(axis=2), 1.0, atol=1e-13)
    for i in range(len(tokens)):
        a = od.anchor_of(out.xattn[i])
        assert a.frame == int(np.argmax(ref[i]))
        assert abs(a.peak - ref[i].max()) < 1e-13


def test_verify_with_anchor_reads_the_last_verified_row(tiny):
    cfg, params, enc = tiny
    model = od.Model(cfg, params)
    st = od.new_state(model, od.cross_kv(model, enc), 7)
    y, _, _ = od.ar_decode(model, st, 4)
    for drafts in ([], [y[0]], [y[0], y[1], (y[2] + 1) % cfg.vocab], y[:3]):
        r, anc = od.verify_with_anchor(model, st, drafts, layer=1)
        ref = od.verify(model, st, drafts)
        assert (r.greedy, r.accepted, r.emitted) == (ref.greedy, ref.accepted, ref.emitted)
        out = od.forward_block(model, st, [st.t0] + list(drafts), probe_layer=1)
        np.testing.assert_array_equal(anc.mean, out.xattn[r.accepted].mean(axis=0))


def test_constructed_weights_closed_forms():
    # q = 8 e_0 makes the score of frame t equal K[t, h, 0]; keys ln(w) give weights w
    w0 = np.array([0.5, 0.4, 0.1])
    w1 = np.array([0.1, 0.5, 0.4])
    K = np.zeros((3, 2, 64))
    K[:, 0, 0], K[:, 1, 0] = np.log(w0), np.log(w1)
    q = np.zeros((1, 2, 64))
    q[0, :, 0] = 8.0
    P = od.attention_probs(q, K, [3])
    np.testing.assert_allclose(P[0], [w0, w1], atol=1e-15)
    a = od.anchor_of(P[0])
    assert a.frame == 1 and abs(a.peak - 0.45) < 1e-15 and abs(a.margin - 0.15) < 1e-15
    # head 0 alone would pick frame 0: the readout averages before the peak
    assert od.anchor_of(P[0, :1]).frame == 0
    # equal keys: uniform weights, the lowest frame wins the tie
    a = od.anchor_of(od.attention_probs(q, np.ones((5, 2, 64)), [5])[0])
    assert a.frame == 0 and abs(a.peak - 0.2) < 1e-15 and a.margin == 0.0
    # one frame: weight 1
    a = od.anchor_of(od.attention_probs(q, K[:1], [1])[0])
    assert a.frame == 0 and a.peak == 1.0
