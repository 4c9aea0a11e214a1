"""Pins for the oracle's sublayers against library routines and closed forms (CPU only)."""
import numpy as np
import torch
import torch.nn.functional as Fn

from oracle.accept import accept_length, argmax_lowest, committed_length, emitted_tokens, top2_margin
from oracle.decoder import attention, gelu, layer_norm, softmax


def test_layer_norm_matches_torch():
    g = np.random.default_rng(0)
    x = g.standard_normal((7, 384)) * 3 + 0.5
    w, b = 1 + 0.02 * g.standard_normal(384), 0.02 * g.standard_normal(384)
    ref = Fn.layer_norm(torch.from_numpy(x), (384,), torch.from_numpy(w), torch.from_numpy(b),
                        eps=1e-5).numpy()
    np.testing.assert_allclose(layer_norm(x, w, b), ref, rtol=0, atol=1e-12)


def test_gelu_matches_torch_and_closed_forms():
    u = np.linspace(-8, 8, 4001)
    ref = Fn.gelu(torch.from_numpy(u), approximate="none").numpy()
    np.testing.assert_allclose(gelu(u), ref, rtol=0, atol=1e-14)
    assert gelu(np.array([0.0]))[0] == 0.0
    # GELU(u) - GELU(-u) = u (Phi(u) + Phi(-u) = 1)
    np.testing.assert_allclose(gelu(u) - gelu(-u), u, atol=1e-13)


def test_attention_matches_sdpa_causal():
    g = np.random.default_rng(1)
    r, H, n0 = 5, 3, 9
    q = g.standard_normal((r, H, 64))
    K = g.standard_normal((n0 + r, H, 64))
    V = g.standard_normal((n0 + r, H, 64))
    out = attention(q, K, V, visible=n0 + np.arange(r) + 1)
    # library: rows are queries at positions n0..n0+r-1 over keys 0..n0+r-1
    mask = torch.ones(r, n0 + r, dtype=torch.bool).tril(diagonal=n0)
    ref = Fn.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2), torch.from_numpy(K).permute(1, 0, 2),
        torch.from_numpy(V).permute(1, 0, 2), attn_mask=mask).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_attention_closed_forms():
    g = np.random.default_rng(2)
    q = g.standard_normal((2, 2, 64))
    v = g.standard_normal((1, 2, 64))
    k = g.standard_normal((1, 2, 64))
    # one key: the output is that key's value
    np.testing.assert_allclose(attention(q, k, v, [1, 1]), np.broadcast_to(v, (2, 2, 64)), atol=1e-15)
    # identical keys: the output is the mean of the values
    K = np.broadcast_to(k, (6, 2, 64))
    V = g.standard_normal((6, 2, 64))
    np.testing.assert_allclose(attention(q, K, V, [6, 6])[0], V.mean(axis=0), atol=1e-13)
    # masked keys never matter, however large
    V2 = V.copy()
    V2[4:] = 1e30
    np.testing.assert_array_equal(attention(q, K, V2, [4, 4]), attention(q, K[:4], V[:4], [4, 4]))


def test_softmax_shift_invariance_and_sum():
    g = np.random.default_rng(3)
    s = g.standard_normal((4, 30)) * 10
    p = softmax(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-14)
    np.testing.assert_allclose(softmax(s + 123.0), p, atol=1e-14)


def test_argmax_lowest_index_and_margin():
    v = np.array([0.5, 2.0, -1.0, 2.0, 1.0])
    assert argmax_lowest(v) == 1
    assert top2_margin(v) == 0.0
    assert top2_margin(np.array([3.0, 1.0, 2.5])) == 0.5


def test_accept_scan_exhaustive():
    # every match/mismatch pattern for k <= 8: a is the number of leading matches
    for k in range(0, 9):
        for pattern in range(1 << k):
            match = [(pattern >> i) & 1 == 1 for i in range(k)]
            greedy = list(range(100, 100 + k + 1))
            drafts = [greedy[i] if match[i] else greedy[i] + 1 for i in range(k)]
            expect = next((j for j in range(k) if not match[j]), k)
            a = accept_length(drafts, greedy)
            assert a == expect
            assert emitted_tokens(greedy, a) == greedy[: a + 1]
            assert committed_length(10, a) == 10 + a + 1


def test_accept_closed_forms():
    g = [5, 6, 7, 8]
    assert accept_length([], [5]) == 0                  # k = 0: an AR step
    assert accept_length([6, 7, 8], g) == 0             # d_1 != g_0
    assert accept_length([5, 6, 7], g) == 3             # all agree: a = k, k + 1 tokens
    assert emitted_tokens(g, 3) == g
