"""Shared pieces of the GPU parity tests: build a device session and the matching oracle
states from the same seeded inputs, and compare outputs.

The parity bar: accept lengths, emitted tokens and KV lengths bit-exact, except at
positions whose oracle top-2 logit margin is below 1e-3; logits within 2e-2 (bf16
storage) or 1e-4 (float32 storage).
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import decoder as od
from paper_2608_12703_amd import ad, synth
from paper_2608_12703_amd.harness import Session

MARGIN_EXCLUDE = 1e-3
KV_EXACT = []          # bit-equal fractions seen by kv_close (reported by the tests)
KV_STATS = []          # (what, layer, sigma, max |diff| / rms, excess over one ulp / rms,
                       #  bit-equal fraction, mean |diff| / rms)
LOGIT_TOL = {"bf16": 2e-2, "f32": 1e-4}


def oracle_model(cfg, params):
    return od.Model(cfg, params)


def oracle_state(cfg, model, b, n, T, t0):
    cross = od.cross_kv(model, synth.make_encoder(cfg, b, T))
    return od.new_state(model, cross, t0, synth.make_prefix_kv(cfg, b, n))


def subset(wl, ids):
    """The workload of the listed sequences only (their own seeded inputs)."""
    ids = list(ids)
    return synth.StepWorkload(wl.k[ids], wl.n[ids], wl.T[ids], wl.t0[ids], wl.G[ids],
                              [wl.fill_ne[i] for i in ids], [wl.fill_any[i] for i in ids])


def device_session(cfg, params, wl, *, layout=ad.AD_PADDED, packed_encoder=False,
                   want_logits=True, poison=False, k_max=None, seq_ids=None, max_frames=1500):
    """Device state for workload `wl`; sequence b draws the inputs of seq_ids[b]."""
    k_max = int(wl.k.max()) if k_max is None else k_max
    ids = list(range(wl.batch)) if seq_ids is None else list(seq_ids)
    s = Session(cfg, params, wl.batch, k_max, wl.T, layout=layout,
                packed_encoder=packed_encoder, want_logits=want_logits, max_frames=max_frames)
    if poison:
        s.pool.fill_(float("nan"))
        s.cross.fill_(float("nan"))
    s.prefill_encoder([synth.make_encoder(cfg, ids[b], int(wl.T[b])) for b in range(wl.batch)])
    for b in range(wl.batch):
        s.import_prefix(b, synth.make_prefix_kv(cfg, ids[b], int(wl.n[b])))
    s.set_kv_len(wl.n)
    return s


def planted_blocks(cfg, model, wl, seqs):
    """Per sequence [t0, d_1..d_k]: oracle-planted drafts for `seqs`, uniform elsewhere."""
    blocks, states = [], {}
    for b in range(wl.batch):
        k = int(wl.k[b])
        if b in seqs:
            st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
            y, _, _ = od.ar_decode(model, st, k)
            d = synth.plant_drafts(np.array(y), int(wl.G[b]), wl.fill_ne[b], wl.fill_any[b])
            states[b] = st
        else:
            d = wl.fill_any[b]
        blocks.append(np.concatenate([[wl.t0[b]], d]).astype(np.int64))
    return blocks, states


def _cross_index():
    """Positions of (frame t, lane j) of a 32-frame block inside its 2048 keys and its
    2048 values: the cross-K/V cache's block layout (the attention operands' order)."""
    t = np.arange(32)[:, None]
    j = np.arange(64)[None, :]
    c16 = 4 * (t // 8) + (t & 3)
    tt = (t // 4) & 1
    k_idx = ((tt * 2 + ((j // 8) & 1)) * 64 + (j // 16) * 16 + c16) * 8 + (j & 7)
    v_idx = ((j // 16) * 64 + (t // 8) * 16 + (j & 15)) * 8 + (t & 7)
    return k_idx, v_idx


def decode_cross(flat: np.ndarray, L: int, H: int, frames_cap: int):
    """[L][H][frames_cap][64] keys and values from a cross-K/V cache array."""
    blk = np.asarray(flat).reshape(L, H, frames_cap // 32, 2, 2048)
    k_idx, v_idx = _cross_index()
    K = blk[:, :, :, 0][..., k_idx].reshape(L, H, frames_cap, 64)
    V = blk[:, :, :, 1][..., v_idx].reshape(L, H, frames_cap, 64)
    return K, V


def encode_cross(K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """The inverse of decode_cross: [L][H][frames_cap][64] keys / values -> cache array."""
    L, H, F, _ = K.shape
    k_idx, v_idx = _cross_index()
    out = np.zeros((L, H, F // 32, 2, 2048), np.float32)
    kb = K.reshape(L, H, F // 32, 32, 64)
    vb = V.reshape(L, H, F // 32, 32, 64)
    out[:, :, :, 0][..., k_idx] = kb
    out[:, :, :, 1][..., v_idx] = vb
    return out.reshape(-1)


def activation_error(gpu_rows, want_rows) -> float:
    """Relative rms error of activation rows against the oracle's: rms(gpu - want) over
    the rms of the oracle's rows centred per row (LayerNorm removes the row mean, so this
    is the relative error a LayerNorm output inherits)."""
    want = np.asarray(want_rows, np.float64)
    c = want - want.mean(axis=-1, keepdims=True)
    d = np.asarray(gpu_rows, np.float64) - want
    return float(np.sqrt(np.mean(d ** 2)) / (np.sqrt(np.mean(c ** 2)) + 1e-30))


def step_taps(sess, blocks, layout=None, parents=None):
    """The residual stream after layers 0 .. L-2 (each the next layer's input) at every
    row of the step: the step is run again with three taps at a time.  It is
    deterministic, so each run rewrites the same outputs and cache bits.  Returns
    {layer: [rows, d] float32}; the session is left prepared as before."""
    L, d = sess.cfg.n_layers, sess.cfg.d_model
    saved = (sess.tap_layers, sess.out_taps)
    sess.out_taps = torch.empty(3, sess.max_rows, d, dtype=torch.float32, device=sess.device)
    out = {}
    layers = list(range(L - 1))
    for i in range(0, len(layers), 3):
        grp = layers[i:i + 3]
        sess.tap_layers = tuple(grp + [-1] * (3 - len(grp)))
        sess.prepare(blocks, layout, parents)
        sess.run()
        t = sess.out_taps.cpu().numpy()
        for j, layer in enumerate(grp):
            out[layer] = t[j, : sess.rows].copy()
    sess.tap_layers, sess.out_taps = saved
    sess.prepare(blocks, layout, parents)
    return out


def layer_input_errors(gpu_taps, ref_taps, rows, L):
    """eps_l for l = 0 .. L-1: the relative error of layer l's input rows (0 for layer 0,
    whose input, the embedding, is the same bf16 sum on both sides)."""
    return [0.0] + [activation_error(gpu_taps[l - 1][rows], ref_taps[l - 1]) for l in range(1, L)]


def compare_sequence(cfg, sess, res, b, block, ref: od.VerifyOut, n: int, check_kv=True,
                     gpu_taps=None):
    """Assert the parity bar for sequence b (committed length n before the step).

    For the cache values, gpu_taps (step_taps) and ref.taps (the oracle's residual
    stream after layers 0 .. L-2) give each layer's input error.  Returns the largest
    logit error."""
    k = len(block) - 1
    rows = [sess.row_of(b, i) for i in range(k + 1)]
    err = 0.0
    if "logits" in res:
        err = float(np.max(np.abs(res["logits"][rows] - ref.logits)))
        print(f"  seq {b}: max logit error {err:.3e}, oracle margins {np.round(ref.margins, 4).tolist()}")
        assert err <= LOGIT_TOL[cfg.dtype], f"seq {b}: logit error {err}"
    g = res["greedy"][rows]
    for i in range(k + 1):
        if ref.margins[i] >= MARGIN_EXCLUDE:
            assert g[i] == ref.greedy[i], \
                f"seq {b} row {i}: greedy {g[i]} vs {ref.greedy[i]} (margin {ref.margins[i]})"
    # the accept decision reads rows 0..a; compare it when none of them is excluded
    a = ref.accepted
    if all(ref.margins[i] >= MARGIN_EXCLUDE for i in range(a + 1)):
        assert res["accept_len"][b] == a, f"seq {b}: accept {res['accept_len'][b]} vs {a}"
        toks = res["out_tokens"][b]
        assert list(toks[: a + 1]) == ref.emitted and np.all(toks[a + 1:] == -1)
    if check_kv:
        L = cfg.n_layers
        if L > 1:
            assert gpu_taps is not None and ref.taps is not None and len(ref.taps) == L - 1, \
                "the cache-value bar needs every layer's input (step_taps and oracle taps)"
            eps = layer_input_errors(gpu_taps, ref.taps, rows, L)
        else:
            eps = [0.0]
        kv = sess.export_prefix(b, n + k + 1)
        for layer, (kb, vb) in enumerate(ref.block_kv):
            kv_close(kv[layer, 0, n:], kb, f"seq {b} layer {layer} K", cfg.dtype, layer, eps[layer])
            kv_close(kv[layer, 1, n:], vb, f"seq {b} layer {layer} V", cfg.dtype, layer, eps[layer])
    return err


KV_SIGMAS = 6.5     # Gaussian tail: P(any of ~1e4 values past 6.5 sigma) < 1e-6
KV_MEAN = 1.5       # E|x| = 0.80 sigma for a normal error; this allows 1.9x that
EPS_OWN = 1e-5      # one projection's own relative error: hi/lo operand 2^-17 + float32
                    # accumulation sqrt(K) 2^-24 (K <= 5120: 4.3e-6), rounded up


def kv_close(gpu: np.ndarray, want: np.ndarray, what: str, dtype: str, layer: int, eps: float):
    """Cache values written by the step against the oracle's stored values.

    The parity bar is exact on what decides tokens and cache slots (greedy tokens, accept
    lengths, committed lengths); cache *values* are intermediate activations.  Both sides
    round a pre-rounding value (GPU a, oracle b) to the storage type, and
    |round(a) - round(b)| <= |a - b| + one ulp, so the bar is one ulp of the stored
    value plus a bound on |a - b|:

    bf16, layer 0: both sides start from the same bf16 embeddings and weights; a - b
    comes only from the GPU's own arithmetic (16-bit activation operands, float32
    accumulation), an error of at most EPS_OWN of the values' rms (it scales with the
    terms of the sum, not with the value: a value near zero from cancellation can lie
    several of its own ulps away).  A value changes only when the two straddle a rounding
    boundary (probability ~|a - b| / ulp): |diff| <= one ulp + KV_SIGMAS EPS_OWN rms, and
    at least 99% of the values bit-equal.

    bf16, layer l >= 1: the layer's input rows differ too (earlier layers' one-ulp
    flips, carried through attention and the residual stream).  Keys / values are a
    LayerNorm output times a random N(0, 0.02) matrix, a projection that keeps relative
    rms errors, so a - b has an rms of sigma = eps + EPS_OWN times the values' rms, eps
    being the measured relative error of this layer's (centred) input rows on the same
    sequence.  Bound per value: one ulp + KV_SIGMAS sigma rms.  Mean: for |a - b| << ulp
    the expected rounded difference equals E|a - b| = 0.8 sigma rms, but it comes in whole
    ulps: value v flips with probability q_v ~ 0.8 sigma rms / ulp_v, by ulp_v, so over N
    values the mean has a standard deviation of at most sqrt(0.8 sigma rms sum_v ulp_v) / N
    (large when N is small: a one-row block of a 128-wide model has 128 values per layer,
    and one flip moves their mean by ~4e-5 rms).  Bound: mean |diff| <= KV_MEAN sigma rms
    + 5 such deviations.
    float32: within 1e-5 relative + 1e-6 absolute, the spread of a float32 accumulation
    against a float64 one.
    """
    want = np.asarray(want, np.float64)
    diff = np.abs(gpu.astype(np.float64) - want)
    rms = float(np.sqrt(np.mean(want ** 2)) + 1e-30)
    ulp = np.abs(want) * 2.0 ** -7
    exact = float(np.mean(diff == 0))
    sigma = eps + EPS_OWN
    excess = float(np.max(np.maximum(diff - ulp, 0.0)) / rms)
    KV_STATS.append((what, layer, sigma, float(diff.max() / rms), excess, exact,
                     float(np.mean(diff) / rms)))
    if dtype == "bf16":
        if layer == 0:
            bad = diff > ulp + KV_SIGMAS * EPS_OWN * rms
            assert not np.any(bad), (f"{what}: {int(bad.sum())} layer-0 cache values past one ulp + "
                                     f"{KV_SIGMAS} x {EPS_OWN} rms")
            KV_EXACT.append(exact)
            assert exact >= 0.99, f"{what}: only {exact:.4f} of layer-0 cache values bit-equal"
        else:
            bad = diff > ulp + KV_SIGMAS * sigma * rms
            assert not np.any(bad), (f"{what}: {int(bad.sum())} cache values past one ulp + "
                                     f"{KV_SIGMAS} x {sigma:.2e} rms (largest excess {excess:.2e} rms)")
            dev = np.sqrt(0.8 * sigma * rms * float(np.sum(ulp))) / diff.size
            assert float(np.mean(diff)) <= KV_MEAN * sigma * rms + 5 * dev, \
                (f"{what}: mean difference {np.mean(diff) / rms:.2e} rms against sigma {sigma:.2e} "
                 f"(+ {5 * dev / rms:.2e} for {diff.size} values)")
    else:
        floor = 1e-5 * rms
        bad = diff > np.abs(want) * 1e-5 + 1e-6 + floor
        assert not np.any(bad), f"{what}: {int(bad.sum())} cache values off by more than 1e-5"


def kv_report(tag: str):
    """Print the worst cache-value statistics collected since the last report."""
    if not KV_STATS:
        return
    l0 = [s for s in KV_STATS if s[1] == 0]
    rest = [s for s in KV_STATS if s[1] > 0]
    msg = f"[{tag}] cache values:"
    if l0:
        msg += f" layer 0 min bit-equal {min(s[5] for s in l0):.4f}, max |diff| {max(s[3] for s in l0):.2e} rms;"
    if rest:
        worst = max(rest, key=lambda s: s[4] / max(s[2], 1e-30))
        mean_w = max(rest, key=lambda s: s[6] / max(s[2], 1e-30))
        msg += (f" layers >= 1: largest excess over one ulp {worst[4] / max(worst[2], 1e-30):.2f} sigma rms"
                f" ({worst[0]}, sigma {worst[2]:.2e}), largest mean |diff| "
                f"{mean_w[6] / max(mean_w[2], 1e-30):.2f} sigma rms ({mean_w[0]}), largest sigma "
                f"{max(x[2] for x in rest):.2e}")
    print(msg, flush=True)
    KV_STATS.clear()


# Head-averaged attention weights: the GPU recomputes row a_b's scores in float32 from its
# own queries, which carry the step's activation error.  A weight's relative error is
# about its score's absolute error: scores of these models have a spread of ~0.5, and
# the queries' relative error stays below 1e-3 (the logits of the 32-layer model differ
# from the oracle's by ~1e-3 on an rms of 0.72), so |d score| <~ 5e-4.  Measured on the
# small shapes: 6e-7 of the peak.  float32 models: the float32 accumulation spread.
ANCHOR_REL = {"bf16": 5e-4, "f32": 1e-5}
ANCHOR_STATS = []      # (seq, frame equal, |peak error| / peak, oracle margin / peak)


def compare_anchor(cfg, res, b, ref: od.VerifyOut, anc: od.Anchor):
    """Anchor readout of sequence b against the oracle's (when its accept decision is
    comparable: the readout reads block row a_b).

    The frame must equal the oracle's unless the oracle's top-2 gap is inside the error
    bound; in every case the oracle's weight at the GPU's frame must lie within the bound
    of the maximum, and the GPU's peak must match the oracle's weight at that frame."""
    if int(res["accept_len"][b]) != ref.accepted:
        return False
    f, peak = int(res["anchor"][b]), float(res["anchor_peak"][b])
    tol = ANCHOR_REL[cfg.dtype] * anc.peak
    assert 0 <= f < anc.mean.size, f"seq {b}: anchor frame {f} outside 0..{anc.mean.size - 1}"
    err = abs(peak - anc.mean[f])
    ANCHOR_STATS.append((b, f == anc.frame, err / anc.peak, anc.margin / anc.peak))
    print(f"  seq {b}: anchor gpu {f} oracle {anc.frame} (T {anc.mean.size}), peak {peak:.6e} "
          f"vs {anc.mean[f]:.6e}, oracle margin {anc.margin / anc.peak:.2e} of peak")
    assert err <= tol, f"seq {b}: anchor peak {peak} vs oracle {anc.mean[f]}"
    assert anc.mean[f] >= anc.peak - 2 * tol, f"seq {b}: frame {f} is not a near-maximum"
    if anc.margin > 2 * tol:
        assert f == anc.frame, f"seq {b}: anchor frame {f} vs oracle {anc.frame}"
    return True
