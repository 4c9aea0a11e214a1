"""Pins for the oracle's audio-conditioned draft step (CPU only).

* The draft block, run incrementally over a round with its KV cache and a cross-attention
  window, against torch's pre-LN ``nn.TransformerDecoderLayer`` over the whole round at
  once (causal mask, encoder memory cut to the window), float64.
* The input projections against ``torch.nn.functional.linear``.
* The window: frames outside it can hold anything (NaN) without changing the round.
* The target's residual-stream taps against the outputs of torch's layers.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import decoder as od
from oracle import draft as odr
from paper_2608_12703_amd import synth


def _torch_layer(cfg, p, layer):
    t = lambda n: torch.from_numpy(np.asarray(p[f"l{layer}.{n}"], np.float64))
    mod = torch.nn.TransformerDecoderLayer(cfg.d_model, cfg.n_heads, cfg.d_ffn, dropout=0.0,
                                           activation="gelu", batch_first=True, norm_first=True,
                                           dtype=torch.float64)
    with torch.no_grad():
        mod.self_attn.in_proj_weight.copy_(t("w_qkv")); mod.self_attn.in_proj_bias.copy_(t("b_qkv"))
        mod.self_attn.out_proj.weight.copy_(t("w_o")); mod.self_attn.out_proj.bias.copy_(t("b_o"))
        mod.multihead_attn.in_proj_weight.copy_(torch.cat([t("w_xq"), t("w_xkv")]))
        mod.multihead_attn.in_proj_bias.copy_(torch.cat([t("b_xq"), t("b_xkv")]))
        mod.multihead_attn.out_proj.weight.copy_(t("w_xo")); mod.multihead_attn.out_proj.bias.copy_(t("b_xo"))
        mod.linear1.weight.copy_(t("w_1")); mod.linear1.bias.copy_(t("b_1"))
        mod.linear2.weight.copy_(t("w_2")); mod.linear2.bias.copy_(t("b_2"))
        for i in (1, 2, 3):
            getattr(mod, f"norm{i}").weight.copy_(t(f"ln{i}_g"))
            getattr(mod, f"norm{i}").bias.copy_(t(f"ln{i}_b"))
    return mod.eval()


@pytest.fixture(scope="module")
def setup(tiny_cfg):
    cfg = tiny_cfg.with_(vocab=97, n_layers=3, dtype="bf16")
    tp = synth.make_params(cfg)
    dp = synth.make_draft_params(cfg)
    dcfg = synth.draft_config(cfg)
    enc = synth.make_encoder(cfg, 0, 90)
    bm = odr.block_model(dcfg, tp, dp, kv_dtype="f64")     # float64 caches for the library pins
    dcross = od.cross_kv(bm, enc)
    return cfg, dcfg, tp, dp, enc, bm, dcross


def test_draft_round_matches_torch_decoder_layer(setup):
    cfg, dcfg, tp, dp, enc, bm, dcross = setup
    g = np.random.default_rng(0)
    taps3, hidden = g.standard_normal((3, cfg.d_model)), g.standard_normal(cfg.d_model)
    anchor, K = 47, 5
    r = odr.draft_round(bm, dp, dcross, taps3, hidden, 11, anchor, 90, K)
    lo, hi = odr.window(anchor, 90)
    assert (lo, hi) == (27, 68)
    # the whole round at once in torch: inputs u_j plus the position embedding of j
    pos = np.asarray(tp["pos_emb"], np.float64)[:K]
    x = torch.from_numpy(np.stack(r.inputs) + pos)[None]
    mem = torch.from_numpy(np.asarray(enc, np.float64)[lo:hi])[None]
    causal = torch.nn.Transformer.generate_square_subsequent_mask(K, dtype=torch.float64)
    with torch.no_grad():
        y = _torch_layer(dcfg, dp, 0)(x, mem, tgt_mask=causal, tgt_is_causal=True)[0]
        h = Fn.layer_norm(y, (cfg.d_model,), torch.from_numpy(np.asarray(dp["lnf_g"], np.float64)),
                          torch.from_numpy(np.asarray(dp["lnf_b"], np.float64)), eps=1e-5)
        logits = (h @ torch.from_numpy(np.asarray(tp["tok_emb"], np.float64)).T).numpy()
    np.testing.assert_allclose(np.stack(r.hidden), h.numpy(), rtol=0, atol=1e-11)
    assert r.drafts == [int(np.argmax(od.round_f32(v))) for v in logits]


def test_draft_round_recursion(setup):
    """The step-to-step wiring of a draft round (EAGLE-3 style, section 3 "Models and
    Protocol"; appendix "Draft architecture"): step 0 reads the fused target feature and
    the pending token; step j >= 1 reads the block's own output of step j - 1 and the
    draft it produced.  Every block input is recomputed with torch ``linear`` from the
    round's recorded outputs; a round that kept the fused feature (or the first token)
    at every step would give different inputs."""
    cfg, dcfg, tp, dp, enc, bm, dcross = setup
    g = np.random.default_rng(3)
    taps3, hidden = g.standard_normal((3, cfg.d_model)), g.standard_normal(cfg.d_model)
    token, anchor, K = 29, 40, 5
    r = odr.draft_round(bm, dp, dcross, taps3, hidden, token, anchor, 90, K)
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    E = T(tp["tok_emb"])
    f0 = Fn.linear(T(np.concatenate([taps3.reshape(-1), hidden])), T(dp["w_fuse"]), T(dp["b_fuse"]))
    feats = [f0] + [T(h) for h in r.hidden[:-1]]
    toks = [token] + r.drafts[:-1]
    for j in range(K):
        u = Fn.linear(torch.cat([feats[j], E[toks[j]]]), T(dp["w_in"]), T(dp["b_in"]))
        np.testing.assert_allclose(r.inputs[j], u.numpy(), rtol=0, atol=1e-12)
        if j >= 1:
            stale = Fn.linear(torch.cat([f0, E[toks[j]]]), T(dp["w_in"]), T(dp["b_in"]))
            assert np.abs(r.inputs[j] - stale.numpy()).max() > 1e-6
    # the drafts are the LM-head argmax of each step's output (the tied token table)
    for j in range(K):
        z = Fn.linear(T(r.hidden[j]), E).numpy()
        assert r.drafts[j] == int(np.argmax(od.round_f32(z)))


def test_input_projections_match_torch_linear(setup):
    cfg, dcfg, tp, dp, enc, bm, dcross = setup
    g = np.random.default_rng(1)
    taps3, hidden = g.standard_normal((3, cfg.d_model)), g.standard_normal(cfg.d_model)
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    f_ref = Fn.linear(T(np.concatenate([taps3.reshape(-1), hidden])), T(dp["w_fuse"]), T(dp["b_fuse"]))
    f = odr.fuse(dp, taps3, hidden)
    np.testing.assert_allclose(f, f_ref.numpy(), rtol=0, atol=1e-12)
    u_ref = Fn.linear(torch.cat([T(f), T(tp["tok_emb"])[42]]), T(dp["w_in"]), T(dp["b_in"]))
    np.testing.assert_allclose(odr.block_input(dp, tp["tok_emb"], f, 42), u_ref.numpy(), rtol=0, atol=1e-12)


def test_frames_outside_the_window_never_matter(setup):
    cfg, dcfg, tp, dp, enc, bm, dcross = setup
    g = np.random.default_rng(2)
    taps3, hidden = g.standard_normal((3, cfg.d_model)), g.standard_normal(cfg.d_model)
    for anchor in (0, 5, 60, 89):
        r = odr.draft_round(bm, dp, dcross, taps3, hidden, 3, anchor, 90, 4)
        lo, hi = odr.window(anchor, 90)
        K, V = dcross[0]
        K2, V2 = K.copy(), V.copy()
        K2[:lo] = K2[hi:] = np.nan
        V2[:lo] = V2[hi:] = np.nan
        r2 = odr.draft_round(bm, dp, [(K2, V2)], taps3, hidden, 3, anchor, 90, 4)
        assert r2.drafts == r.drafts
        np.testing.assert_array_equal(np.stack(r2.hidden), np.stack(r.hidden))
    # a different centre changes the audio the draft sees
    assert odr.window(0, 90) == (0, 21) and odr.window(89, 90) == (69, 90)


def test_target_taps_are_the_layer_outputs(setup):
    cfg, dcfg, tp, dp, enc, bm, dcross = setup
    model = od.Model(cfg, tp, kv_dtype="f64")
    tokens = [5, 17, 3, 3, 96]
    out = od.forward_block(model, od.new_state(model, od.cross_kv(model, enc), tokens[0]), tokens,
                           taps=odr.tap_layers(cfg.n_layers))
    assert odr.tap_layers(cfg.n_layers) == [0, 0, 1]
    t = lambda name: torch.from_numpy(np.asarray(tp[name], np.float64))
    x = (t("tok_emb")[torch.tensor(tokens)] + t("pos_emb")[: len(tokens)])[None]
    mem = torch.from_numpy(np.asarray(enc, np.float64))[None]
    causal = torch.nn.Transformer.generate_square_subsequent_mask(len(tokens), dtype=torch.float64)
    outs = []
    with torch.no_grad():
        for layer in range(cfg.n_layers):
            x = _torch_layer(cfg, tp, layer)(x, mem, tgt_mask=causal, tgt_is_causal=True)
            outs.append(x[0].numpy())
    for i, layer in enumerate(odr.tap_layers(cfg.n_layers)):
        np.testing.assert_allclose(out.taps[i], outs[layer], rtol=0, atol=1e-11)
