"""The encoder K/V prefill (setup, once per utterance: the decoder reuses the encoded
audio at every step) against the oracle's projection, value by value.

K_l = enc W_k,l^T and V_l = enc W_v,l^T + b_v,l in float64, rounded to bf16, against the
cache the matrix-core prefill writes (decoded from the cache's 32-frame block layout).
Both sides round the same d-term sum (float32 matrix accumulation on the GPU, float64
in the oracle) to bf16.  The two sums differ by ~1e-6 of the values' rms (an error that
scales with the terms, so a value near zero may lie several of its own ulps away), far
below an ulp of 2^-8..2^-7 of a typical value: a value differs only when the sums
straddle a rounding boundary.  Bar: one ulp + KV_SIGMAS EPS_OWN rms everywhere (the
cache-value bar of the step's first layer) and at least 99.9% of the values bit-equal.
float32 models (the VALU prefill): 1e-5 relative."""
import numpy as np
import pytest

from oracle import decoder as od
from paper_2608_12703_amd import synth
from paper_2608_12703_amd.configs import CONFIGS, Config
from paper_2608_12703_amd.harness import Session

from gpu_common import EPS_OWN, KV_SIGMAS, decode_cross

pytestmark = pytest.mark.gpu


def _check(cfg, frames, layers, seq_ids=None, pack_weights=True):
    params = synth.make_params(cfg)
    B = len(frames)
    ids = list(range(B)) if seq_ids is None else seq_ids
    sess = Session(cfg, params, B, 0, frames, pack_weights=pack_weights)
    encs = [synth.make_encoder(cfg, ids[b], frames[b]) for b in range(B)]
    sess.prefill_encoder(encs)
    flat = sess.cross.float().cpu().numpy()
    K, V = decode_cross(flat, cfg.n_layers, cfg.n_heads, sess.frames_cap)
    offs = sess.enc_off.cpu().numpy()
    model = od.Model(cfg, {n: params[n] for n in params})
    worst, exact = 0.0, []
    for b in range(B):
        ref = od.cross_kv(model, encs[b])          # per layer (K, V) [T, H, 64], stored
        sl = slice(int(offs[b]), int(offs[b]) + frames[b])
        for layer in layers:
            for got, want in ((K[layer][:, sl].transpose(1, 0, 2), ref[layer][0]),
                              (V[layer][:, sl].transpose(1, 0, 2), ref[layer][1])):
                want = np.asarray(want, np.float64)
                diff = np.abs(got.astype(np.float64) - want)
                rms = float(np.sqrt(np.mean(want ** 2)))
                if cfg.dtype == "bf16":
                    bad = diff > np.abs(want) * 2.0 ** -7 + KV_SIGMAS * EPS_OWN * rms
                    assert not np.any(bad), f"seq {b} layer {layer}: {int(np.sum(bad))} values past the bar"
                    exact.append(float(np.mean(diff == 0)))
                else:
                    assert np.all(diff <= np.abs(want) * 1e-5 + 1e-6)
                worst = max(worst, float(diff.max()))
    if exact:
        print(f"[{cfg.name}] prefill: largest difference {worst:.3e}, least bit-equal fraction {min(exact):.5f}")
        assert min(exact) >= 0.999
    return sess


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_prefill_matches_oracle_small(dtype):
    cfg = Config(name="unit_prefill", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
                 dtype=dtype, batch=3, k=1, frames=300, seed=5)
    # ragged lengths: tails inside a 32-frame block and inside a 256-frame tile
    _check(cfg, [300, 37, 129], layers=[0, 1])


@pytest.mark.parametrize("pack_weights", [True, False])
@pytest.mark.parametrize("n_layers", [1, 3])
def test_prefill_operand_layouts(pack_weights, n_layers):
    """Tiled and row-major weights; one layer (the encoder states are read row-major) and
    three (the first two read them in fragment order, staged in the last layer's cache).
    d 512: whole 256-column key and value tiles (the 8-byte stores) next to a frame tail."""
    cfg = Config(name="unit_prefill_layout", n_layers=n_layers, d_model=512, n_heads=8, d_ffn=1024,
                 vocab=1000, dtype="bf16", batch=2, k=1, frames=600, seed=9)
    _check(cfg, [600, 211], layers=list(range(n_layers)), pack_weights=pack_weights)


def test_prefill_matches_oracle_large_v3():
    """The bench's shape: 1500 frames, d 1280, 20 heads; four layers of two utterances
    (the oracle's float64 projection of every layer would take a minute)."""
    cfg = CONFIGS["large_v3_bf16"]
    _check(cfg, [1500, 1500], layers=[0, 9, 20, 31], seq_ids=[0, 17])
