"""Pins for the oracle's AnchorDraft objective (CPU only).

Paper, section "Correction and Cost", paragraph "AnchorDraft Training Objective", and
appendix "Training Correction with AnchorDraft" (eq. anchordraft-supp).
* q_t: sums to 1 over the valid keys; its normaliser far from the edges is the
  Gaussian integral sigma sqrt(2 pi) (Poisson summation: the correction is e^-493 at
  sigma = 5); a tiny sigma gives the one-hot target, so l_t = -log Abar_t(c_t).
* l_t = H(q_t) + KL(q_t || Abar_t), with both computed by scipy.stats.entropy (so a
  wrong sign, log base, normalisation or dropped term fails); the minimum H(q_t) is
  reached when the head-averaged attention equals q_t (keys built so that softmax = q),
  and there the gradient vanishes.
* The gradient with respect to the query rows against central finite differences of
  the loss, and against torch autograd of an independent float64 expression.
* Masking: padded keys (NaN) never matter; unaligned rows add nothing and do not count.
* Head averaging: H copies of one head give that head's loss; permuting heads changes
  nothing.
* L_tok and L_feat and their gradients against torch's cross_entropy (ignore_index) and
  smooth_l1_loss (beta = 1) with autograd.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn
from scipy.stats import entropy

from oracle import anchor_loss as al


def _case(seed, r=6, H=3, T=70, T_cap=80):
    g = np.random.default_rng(seed)
    xq = g.standard_normal((r, H * 64))
    K = g.standard_normal((T_cap, H, 64)) * 0.3
    cen = g.integers(0, T, r)
    return xq, K, T, cen


def test_gaussian_target():
    for c in (0, 7, 59):
        q = al.gaussian_target(c, 60, 5.0)
        assert abs(q.sum() - 1.0) < 1e-15 and np.argmax(q) == c
        assert np.all(q > 0)
    # normaliser in the interior: sigma sqrt(2 pi)
    j = np.arange(400, dtype=np.float64)
    z = np.sum(np.exp(-((j - 200) ** 2) / 50.0))
    assert abs(z / (5.0 * np.sqrt(2 * np.pi)) - 1.0) < 1e-14
    q = al.gaussian_target(200, 400, 5.0)
    np.testing.assert_allclose(q[200], 1.0 / (5.0 * np.sqrt(2 * np.pi)), rtol=1e-14)
    # symmetric about an interior centre, truncated and renormalised at the edge
    np.testing.assert_allclose(q[190:200], q[210:200:-1], rtol=1e-14)
    q0 = al.gaussian_target(0, 400, 5.0)
    half = np.sum(np.exp(-(np.arange(0, 400.0) ** 2) / 50.0))
    np.testing.assert_allclose(q0[0], 1.0 / half, rtol=1e-15)
    np.testing.assert_allclose(half, 5.0 * np.sqrt(2 * np.pi) / 2 + 0.5, rtol=1e-14)


def test_row_loss_is_entropy_plus_kl():
    xq, K, T, cen = _case(0)
    out = al.anchor_loss([xq], [K], [T], [cen])
    A = al.cross_attention_probs(xq, K, T)
    for t, c in enumerate(cen):
        q = al.gaussian_target(int(c), T, 5.0)
        abar = A[t].mean(axis=0)
        want = entropy(q) + entropy(q, abar)
        np.testing.assert_allclose(out.row_loss[0][t], want, rtol=1e-12)
        assert out.row_loss[0][t] >= entropy(q)
    assert out.n_valid == len(cen)
    np.testing.assert_allclose(out.loss, np.mean(out.row_loss[0]), rtol=1e-14)


def test_minimum_at_the_gaussian():
    # one head, keys along one axis: score_j = log q(j), so softmax = q exactly
    T, c = 50, 21
    q = al.gaussian_target(c, T, 5.0)
    K = np.zeros((T, 1, 64))
    K[:, 0, 0] = np.log(q)
    xq = np.zeros((1, 64))
    xq[0, 0] = 8.0
    out = al.anchor_loss([xq], [K], [T], [np.array([c])])
    np.testing.assert_allclose(out.abar[0][0], q, rtol=1e-12)
    np.testing.assert_allclose(out.loss, entropy(q), rtol=1e-12)
    assert np.max(np.abs(out.dxq[0])) < 1e-12
    # a one-hot target (tiny sigma): l = -log Abar(c)
    xq2, K2, T2, cen2 = _case(1, r=2)
    out2 = al.anchor_loss([xq2], [K2], [T2], [cen2], sigma=0.05)
    for t in range(2):
        np.testing.assert_allclose(out2.row_loss[0][t], -np.log(out2.abar[0][t][cen2[t]]), rtol=1e-12)


def test_gradient_against_finite_differences_and_autograd():
    xq, K, T, cen = _case(2, r=3, H=2, T=40)
    cen[1] = -1
    out = al.anchor_loss([xq], [K], [T], [cen], lam=0.1)
    f = lambda x: 0.1 * al.anchor_loss([x], [K], [T], [cen]).loss
    g = np.random.default_rng(9)
    for _ in range(12):
        t, i = int(g.integers(0, 3)), int(g.integers(0, 128))
        e = np.zeros_like(xq)
        e[t, i] = 1e-5
        fd = (f(xq + e) - f(xq - e)) / 2e-5
        assert abs(fd - out.dxq[0][t, i]) < 1e-8 + 1e-6 * abs(fd)
    # autograd of a float64 torch expression written independently
    x = torch.tensor(xq, dtype=torch.float64, requires_grad=True)
    k = torch.tensor(K[:T], dtype=torch.float64)
    s = torch.einsum("rhd,jhd->rhj", x.view(3, 2, 64), k) / 8
    abar = torch.softmax(s, dim=-1).mean(dim=1)
    tot = 0
    for t in (0, 2):
        j = torch.arange(T, dtype=torch.float64)
        w = torch.exp(-(j - int(cen[t])) ** 2 / 50.0)
        tot = tot - (w / w.sum() * torch.log(abar[t])).sum()
    (0.1 * tot / 2).backward()
    np.testing.assert_allclose(out.dxq[0], x.grad.numpy(), rtol=1e-9, atol=1e-14)
    assert np.all(out.dxq[0][1] == 0)


def test_masking():
    xq, K, T, cen = _case(3)
    out = al.anchor_loss([xq], [K], [T], [cen])
    K2 = K.copy()
    K2[T:] = np.nan
    out2 = al.anchor_loss([xq], [K2], [T], [cen])
    np.testing.assert_array_equal(out.row_loss[0], out2.row_loss[0])
    np.testing.assert_array_equal(out.dxq[0], out2.dxq[0])
    # an unaligned row contributes nothing and is not counted
    xq3 = np.concatenate([xq, np.ones((1, xq.shape[1]))])
    out3 = al.anchor_loss([xq3], [K], [T], [np.concatenate([cen, [-1]])])
    assert out3.n_valid == out.n_valid and out3.row_loss[0][-1] == 0
    np.testing.assert_allclose(out3.loss, out.loss, rtol=1e-15)
    # two sequences: |V| counts the aligned rows of the batch
    xb, Kb, Tb, cb = _case(4, r=4, T=33, T_cap=40)
    both = al.anchor_loss([xq, xb], [K, Kb], [T, Tb], [cen, cb])
    one = al.anchor_loss([xb], [Kb], [Tb], [cb])
    np.testing.assert_allclose(both.loss * 10, out.loss * 6 + one.loss * 4, rtol=1e-13)


def test_head_averaging():
    xq, K, T, cen = _case(5, H=1)
    out1 = al.anchor_loss([xq], [K], [T], [cen])
    xq3 = np.tile(xq, (1, 3))
    K3 = np.repeat(K, 3, axis=1)
    out3 = al.anchor_loss([xq3], [K3], [T], [cen])
    np.testing.assert_allclose(out3.row_loss[0], out1.row_loss[0], rtol=1e-13)
    xq, K, T, cen = _case(6, H=4)
    perm = [2, 0, 3, 1]
    xp = xq.reshape(len(cen), 4, 64)[:, perm].reshape(len(cen), -1)
    outp = al.anchor_loss([xp], [K[:, perm]], [T], [cen])
    np.testing.assert_allclose(outp.row_loss[0], al.anchor_loss([xq], [K], [T], [cen]).row_loss[0], rtol=1e-13)


def test_token_and_feature_terms_against_torch():
    g = np.random.default_rng(7)
    z = g.standard_normal((9, 31)) * 3
    y = g.integers(0, 31, 9)
    y[[2, 5]] = -1
    loss, dz = al.token_loss(z, y)
    zt = torch.tensor(z, requires_grad=True)
    ref = Fn.cross_entropy(zt, torch.tensor(y), ignore_index=-1)
    ref.backward()
    np.testing.assert_allclose(loss, ref.item(), rtol=1e-13)
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-16)
    p, tgt = g.standard_normal((9, 16)) * 2, g.standard_normal((9, 16))
    valid = y >= 0
    lf, dp = al.feature_loss(p, tgt, valid)
    pt = torch.tensor(p, requires_grad=True)
    reff = Fn.smooth_l1_loss(pt[torch.tensor(valid)], torch.tensor(tgt)[torch.tensor(valid)], beta=1.0)
    reff.backward()
    np.testing.assert_allclose(lf, reff.item(), rtol=1e-13)
    np.testing.assert_allclose(dp, pt.grad.numpy(), rtol=1e-12, atol=1e-16)
    # the objective's weights: L = L_tok + 0.5 L_feat + lambda L_anchor
    xq, K, T, cen = _case(8, r=9)
    o = al.objective(z, y, p, tgt, [xq], [K], [T], [cen], lam=0.1)
    np.testing.assert_allclose(o.total, loss + 0.5 * lf + 0.1 * o.anchor, rtol=1e-14)
    np.testing.assert_allclose(o.dfeat, 0.5 * dp, rtol=0)
