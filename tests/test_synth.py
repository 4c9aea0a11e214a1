"""Host-side checks of the seeded input generators (CPU only)."""
import numpy as np

from oracle.accept import accept_length
from paper_2608_12703_amd import configs, synth


def test_params_are_seeded_bf16_and_keyless_bias(tiny_cfg):
    p1 = synth.make_params(tiny_cfg)
    p2 = synth.make_params(tiny_cfg)
    for name, shape in synth.param_specs(tiny_cfg):
        assert p1[name].shape == shape
        np.testing.assert_array_equal(p1[name], p2[name])
        assert np.all((p1[name].view(np.uint32) & 0xFFFF) == 0)      # bf16-representable
    d = tiny_cfg.d_model
    assert np.all(p1["l0.b_qkv"][d:2 * d] == 0) and np.all(p1["l1.b_xkv"][:d] == 0)
    assert abs(float(np.mean(p1["l0.ln1_g"])) - 1.0) < 0.01
    assert len(synth.param_specs(tiny_cfg)) == 4 + 20 * tiny_cfg.n_layers


def test_sequence_inputs_do_not_depend_on_batch():
    cfg = configs.RAGGED_LARGE_V3
    w8 = synth.make_step_workload(cfg, batch=8)
    w3 = synth.make_step_workload(cfg, batch=3)
    for f in ("k", "n", "T", "t0", "G"):
        np.testing.assert_array_equal(getattr(w8, f)[:3], getattr(w3, f))
    assert np.all((w8.k >= 2) & (w8.k <= 8))
    assert np.all((w8.T >= 200) & (w8.T <= 1500))
    assert np.all(w8.n + w8.k + 1 <= configs.MAX_POS)


def test_planted_drafts_accept_exactly_min_g_k():
    g = np.random.default_rng(0)
    for _ in range(500):
        k = int(g.integers(0, 9))
        y = g.integers(0, 5, size=k + 1)          # small vocab: many accidental repeats
        G = int(g.integers(0, 12))
        d = synth.plant_drafts(y[:k], G, g.integers(0, 4, k), g.integers(0, 5, k))
        assert accept_length(d, y) == min(G, k)


def test_drift_plan_rejects_at_each_anchor():
    cfg = configs.DRIFT_STRESS
    plan = synth.make_drift_plan(cfg, 0)
    assert np.all(np.diff(plan.anchors) >= 1) and set(plan.signs.tolist()) <= {-1, 1}
    g = np.random.default_rng(1)
    y = g.integers(0, 3, size=configs.MAX_POS + 1)   # tiny alphabet: shifted tokens often equal
    n, rounds = 0, 0
    while n <= configs.MAX_POS - 1:
        k = min(cfg.k, configs.MAX_POS - 1 - n)
        d = synth.plant_drift(y, n, k, plan)
        a = accept_length(d, y[n + 1: n + 1 + k])
        nxt = plan.anchors[plan.anchors > n]
        if len(nxt) and nxt[0] <= n + k:
            assert a == nxt[0] - n - 1               # rejected exactly at the anchor
        else:
            assert a == k
        n += a + 1
        rounds += 1
    assert n == configs.MAX_POS and rounds > configs.MAX_POS // (cfg.k + 1)
