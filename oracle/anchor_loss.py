"""AnchorDraft training objective (test infrastructure only).

Paper, section "Correction and Cost", paragraph "AnchorDraft Training Objective"
(eq. anchordraft-main), and appendix "Training Correction with AnchorDraft"
(eq. anchordraft-supp): a training-only loss pulls the draft's first-layer audio
attention towards the forced-alignment frame of the next token,

  Abar_t(j) = (1/H) sum_h A_{t,hj}
  q_t(j)    = exp(-(j - c_t)^2 / (2 sigma^2)) / sum_{l in K_u} exp(-(l - c_t)^2 / (2 sigma^2))
  L         = L_tok + 0.5 L_feat - (lambda / |V|) sum_{t in V} sum_{j in K_u} q_t(j) log Abar_t(j)

with K_u the utterance's valid audio keys and V the positions that have an alignment.
The appendix "Training" paragraph names the other two terms: token cross-entropy and a
smooth-L1 feature loss weighted by 0.5; the selected setting is lambda = 0.1, sigma = 5.

Readings used here (the paper gives the formulas, not the reductions):
* A_{t,hj} is the first draft layer's cross-attention: the softmax over the valid keys
  j = 0 .. T-1 (padded frames excluded) of (x_{t,h} . k_{h,j}) / 8, with x_t the layer's
  cross-attention query row (64-wide heads).
* c_t is an integer frame in 0 .. T-1, or -1 for a position without an alignment (not
  in V).  |V| counts the aligned positions of the whole batch.
* L_tok is the mean over the positions with a next token (target >= 0) of
  logsumexp(z_t) - z_t[y_t]; L_feat is the mean over the elements of those positions
  of smooth-L1 with beta = 1 (0.5 e^2 for |e| < 1, else |e| - 0.5).
* Gradients follow from the definitions: dl_t/dA_{t,hj} = -q_t(j) / (H Abar_t(j)), the
  softmax Jacobian gives dl_t/dS_{t,hj} = A_{t,hj} (g_j - sum_i A_{t,hi} g_i), and
  dl_t/dx_{t,h} = (1/8) sum_j dl_t/dS_{t,hj} k_{h,j}.

Float64 throughout; the inputs are whatever the caller stores (queries, keys, logits).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

HEAD = 64
LAMBDA = 0.1
SIGMA = 5.0


def gaussian_target(center: int, T: int, sigma: float) -> np.ndarray:
    """q(j) over the valid keys j = 0 .. T-1, centred on `center`, summing to 1."""
    j = np.arange(T, dtype=np.float64)
    w = np.exp(-((j - center) ** 2) / (2.0 * sigma * sigma))
    return w / w.sum()


def cross_attention_probs(xq: np.ndarray, K: np.ndarray, T: int) -> np.ndarray:
    """A [r, H, T]: softmax over the valid keys of (x_{t,h} . k_{h,j}) / 8.
    xq: [r, H*64] query rows; K: [>= T, H, 64] (only the first T keys are read)."""
    r = xq.shape[0]
    H = K.shape[1]
    q = np.asarray(xq, np.float64).reshape(r, H, HEAD)
    k = np.asarray(K[:T], np.float64)
    s = np.einsum("rhd,jhd->rhj", q, k) / 8.0
    s -= s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


@dataclass
class AnchorLossOut:
    loss: float                 # lambda-free L_anchor = (1/|V|) sum_t l_t
    n_valid: int                # |V|
    row_loss: list              # per sequence: l_t = -sum_j q_t(j) log Abar_t(j) (0 where unaligned)
    abar: list                  # per sequence: Abar [r_b, T_b]
    dxq: list                   # per sequence: d(lambda L_anchor)/dx [r_b, H*64]


def anchor_loss(xqs, Ks, Ts, centers, sigma: float = SIGMA, lam: float = LAMBDA) -> AnchorLossOut:
    """The alignment term over a batch of utterances: sequence b has query rows xqs[b]
    [r_b, H*64], first-layer cross keys Ks[b] [>= T_b, H, 64], T_b = Ts[b] valid frames
    and per-row centres centers[b] [r_b] (-1: unaligned)."""
    As = [cross_attention_probs(xq, K, int(T)) for xq, K, T in zip(xqs, Ks, Ts)]
    return anchor_loss_from_probs(As, Ks, centers, sigma, lam)


def anchor_loss_from_probs(As, Ks, centers, sigma: float = SIGMA, lam: float = LAMBDA) -> AnchorLossOut:
    """The same from the attention probabilities As[b] [r_b, H, T_b] (the gradient needs
    the keys, not the queries)."""
    n_valid = sum(int(np.sum(np.asarray(c) >= 0)) for c in centers)
    rows, abars, grads = [], [], []
    for A, K, cen in zip(As, Ks, centers):
        A = np.asarray(A, np.float64)
        T = A.shape[2]
        H = A.shape[1]
        abar = A.mean(axis=1)                              # [r, T]
        ell = np.zeros(len(cen))
        dx = np.zeros((len(cen), H * HEAD))
        for t, c in enumerate(cen):
            if c < 0:
                continue
            q = gaussian_target(int(c), T, sigma)
            ell[t] = -np.sum(q * np.log(abar[t]))
            g = -q / (H * abar[t])                         # dl/dA_{hj}, the same for every head
            dS = A[t] * (g[None, :] - np.sum(A[t] * g[None, :], axis=1, keepdims=True))
            dxh = np.einsum("hj,jhd->hd", dS, np.asarray(K[:T], np.float64)) / 8.0
            dx[t] = (lam / max(n_valid, 1)) * dxh.reshape(-1)
        rows.append(ell)
        abars.append(abar)
        grads.append(dx)
    total = sum(float(r.sum()) for r in rows) / max(n_valid, 1)
    return AnchorLossOut(total, n_valid, rows, abars, grads)


def token_loss(logits: np.ndarray, targets) -> tuple[float, np.ndarray]:
    """Mean cross-entropy over the rows with a target >= 0, and its gradient
    d L_tok / d logits."""
    z = np.asarray(logits, np.float64)
    y = np.asarray(targets)
    valid = y >= 0
    n = max(int(valid.sum()), 1)
    m = z.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(z - m).sum(axis=1))
    loss = float(np.sum((lse - z[np.arange(len(y)), np.where(valid, y, 0)])[valid]) / n)
    p = np.exp(z - lse[:, None])
    p[np.arange(len(y)), np.where(valid, y, 0)] -= 1.0
    grad = np.where(valid[:, None], p / n, 0.0)
    return loss, grad


def feature_loss(pred: np.ndarray, target: np.ndarray, valid) -> tuple[float, np.ndarray]:
    """Mean smooth-L1 (beta = 1) over the elements of the valid rows, and its gradient
    d L_feat / d pred."""
    e = np.asarray(pred, np.float64) - np.asarray(target, np.float64)
    valid = np.asarray(valid, bool)
    n = max(int(valid.sum()), 1) * e.shape[1]
    a = np.abs(e)
    per = np.where(a < 1.0, 0.5 * e * e, a - 0.5)
    loss = float(np.sum(per[valid]) / n)
    grad = np.where(valid[:, None], np.clip(e, -1.0, 1.0) / n, 0.0)
    return loss, grad


@dataclass
class ObjectiveOut:
    total: float
    tok: float
    feat: float
    anchor: float               # L_anchor (before lambda)
    anchor_out: AnchorLossOut
    dlogits: np.ndarray         # d total / d logits
    dfeat: np.ndarray           # d total / d predicted features


def objective(logits, targets, pred, feat_target, xqs, Ks, Ts, centers,
              sigma: float = SIGMA, lam: float = LAMBDA) -> ObjectiveOut:
    """L = L_tok + 0.5 L_feat + lambda L_anchor over a batch whose rows are the
    concatenation of the sequences' rows (logits, targets, pred, feat_target: [rows, ..])."""
    tok, dz = token_loss(logits, targets)
    valid = np.asarray(targets) >= 0
    feat, df = feature_loss(pred, feat_target, valid)
    an = anchor_loss(xqs, Ks, Ts, centers, sigma, lam)
    return ObjectiveOut(tok + 0.5 * feat + lam * an.loss, tok, feat, an.loss, an, dz, 0.5 * df)
