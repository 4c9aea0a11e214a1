"""Host-driven speculative decode loops over the C-ABI step (paper, section 3 "Speculative
Loop" and appendix "Real cached loop"): verify a drafted block, commit the accepted
prefix plus the bonus token, draft again.  Every step of the hot path runs in libad;
these loops only move token ids between rounds.

Two drafters:
  * linear draft heads on the final hidden state (ad_draft_heads), the tiny model's
    drafter;
  * planted drafts that follow a known greedy continuation and drift off it by +-1 token
    after anchor points (the drift-stress workload).
"""
from __future__ import annotations

import numpy as np
import torch

from . import ad, synth
from .configs import MAX_POS


def _clamp_k(k: int, n: int) -> int:
    """Draft length that keeps the block inside the learned positions."""
    return max(0, min(k, MAX_POS - 1 - n))


def decode_with_heads(sess, heads_w, t0, n_tokens: int):
    """Greedy speculative decode of every sequence of `sess` for n_tokens tokens.

    heads_w: device tensor [n_heads, vocab, d] of the model dtype.  Round 0 verifies the
    pending token alone (no hidden state exists yet); every later round drafts with the
    heads on the hidden row of the last accepted position.
    Returns (tokens [B][n_tokens], accepts: list of per-round accept arrays,
    drafts: list of per-round draft lists [B][k_b], rounds).
    """
    B, H = sess.B, heads_w.shape[0]
    assert sess.k_max >= H and sess.layout == ad.AD_PADDED
    ws = torch.empty(sess.model.draft_heads_workspace_size(H, B), dtype=torch.uint8,
                     device=sess.device)
    nxt = torch.zeros(B, H + 1, dtype=torch.int32, device=sess.device)
    toks = [[] for _ in range(B)]
    accepts, drafts = [], []
    n = sess.kv_len.cpu().numpy().astype(np.int64)
    blocks = [np.array([int(t0[b])], np.int64) for b in range(B)]
    rounds = 0
    while min(len(t) for t in toks) < n_tokens:
        drafts.append([blk[1:].copy() for blk in blocks])
        sess.step(blocks)
        sess.commit()
        ad.draft_heads(sess.model, heads_w, H, sess.out_hidden, sess.layout, sess.k_max, None,
                       sess.accept_len, sess.out_tokens, B, nxt, ws)
        res = sess.results()
        assert res["err"] == 0, f"device error flag {res['err']}"
        a = res["accept_len"]
        accepts.append(a.copy())
        nt = nxt.cpu().numpy()
        for b in range(B):
            toks[b] += [int(x) for x in res["out_tokens"][b][: a[b] + 1]]
            n[b] += a[b] + 1
            k = _clamp_k(H, int(n[b]))
            blocks[b] = nt[b][: k + 1].astype(np.int64)
        rounds += 1
    return [t[:n_tokens] for t in toks], accepts, drafts, rounds


def decode_with_drift(sess, ys, plans, k: int, n_tokens: int):
    """Speculative decode with drifting planted drafts (synth.plant_drift).

    ys[b] is sequence b's greedy continuation from position 0 (ys[b][0] = the pending
    start token); the committed prefix starts empty.  A sequence that already has
    n_tokens tokens verifies its pending token alone until the others catch up, so ys[b]
    needs n_tokens + k + 1 entries.  Returns (tokens, accepts, rounds).
    """
    B = sess.B
    toks = [[] for _ in range(B)]
    accepts = []
    n = np.zeros(B, np.int64)
    pending = [int(y[0]) for y in ys]     # the step's own bonus token after round 0
    rounds = 0
    done = lambda: min(len(t) for t in toks) >= n_tokens
    while not done():
        blocks = []
        for b in range(B):
            kb = _clamp_k(k, int(n[b])) if len(toks[b]) < n_tokens else 0
            blocks.append(np.concatenate([[pending[b]], synth.plant_drift(ys[b], int(n[b]), kb, plans[b])]))
        sess.step(blocks)
        sess.commit()
        res = sess.results()
        assert res["err"] == 0, f"device error flag {res['err']}"
        a = res["accept_len"]
        accepts.append(a.copy())
        for b in range(B):
            emitted = [int(x) for x in res["out_tokens"][b][: a[b] + 1]]
            toks[b] += emitted
            pending[b] = emitted[-1]
            n[b] += a[b] + 1
        rounds += 1
        if int(n.max()) >= MAX_POS:
            break
    return [t[:n_tokens] for t in toks], accepts, rounds
