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
        res = sess.results(keys=("accept_len", "out_tokens", "err"))
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


def decode_with_drift(sess, ys, plans, k: int, n_tokens: int, ks_out=None):
    """Speculative decode with drifting planted drafts (synth.plant_drift).

    ys[b] is sequence b's greedy continuation from position 0 (ys[b][0] = the pending
    start token); the committed prefix starts empty.  The batch is static: a sequence
    that already has n_tokens tokens stays in it as an idle one-row block (its pending
    token verified again at its last position, nothing kept) until every sequence is
    done.  ys[b] needs min(n_tokens + k, MAX_POS - 1) + 1 entries.  ks_out, if given,
    receives each round's draft lengths ([B] arrays, -1 for an idle sequence).
    Returns (tokens, accepts, rounds).
    """
    B = sess.B
    toks = [[] for _ in range(B)]
    accepts = []
    n = np.zeros(B, np.int64)
    pending = [int(y[0]) for y in ys]     # the step's own bonus token after round 0
    rounds = 0
    done = lambda: min(len(t) for t in toks) >= n_tokens
    while not done():
        # finished sequences re-verify at their last position (the commit's move of
        # their length is undone here each round)
        sess.set_kv_len(np.minimum(n, MAX_POS - 1))
        live = [len(toks[b]) < n_tokens for b in range(B)]
        ks = np.array([_clamp_k(k, int(n[b])) if live[b] else 0 for b in range(B)])
        blocks = [np.concatenate([[pending[b]], synth.plant_drift(ys[b], int(n[b]), int(ks[b]), plans[b])])
                  for b in range(B)]
        sess.step(blocks)
        sess.commit()
        res = sess.results(keys=("accept_len", "out_tokens", "err"))
        assert res["err"] == 0, f"device error flag {res['err']}"
        a = res["accept_len"]
        accepts.append(a.copy())
        if ks_out is not None:
            ks_out.append(np.where(live, ks, -1))
        for b in range(B):
            if not live[b]:
                continue
            emitted = [int(x) for x in res["out_tokens"][b][: a[b] + 1]]
            toks[b] += emitted
            pending[b] = emitted[-1]
            n[b] += a[b] + 1
        rounds += 1
    return [t[:n_tokens] for t in toks], accepts, rounds


# ---------------------------------------------------------------------- audio-conditioned draft

HALF_WINDOW = 20   # frames: +-400 ms at 20 ms per encoder frame


class DraftRunner:
    """The audio-conditioned draft block of a target session: a one-layer model of the
    target's form (its own block and final LayerNorm, the target's token and position
    tables) run through ad_verify_step with one row per sequence, fed by ad_draft_input.

    Rounds start from a target step that was run with anchor_layer >= 0 and three
    tap_layers (see Session); every draft step is a device-side pair of calls.
    """

    def __init__(self, target, draft_params: dict, pack_weights: bool = True):
        from .harness import Session, upload
        cfg, B = target.cfg, target.B
        self.target, self.B = target, B
        self.dcfg = synth.draft_config(cfg)
        dt = target.dt
        dev = target.device
        own = {n: upload(draft_params[n], dt, dev) for n, _ in synth.draft_param_specs(cfg)}
        shared = {"tok_emb": target.params[0], "pos_emb": target.params[1]}
        plist = [shared[n] if n in shared else own[n] for n, _ in synth.param_specs(self.dcfg)]
        self.sess = Session(self.dcfg, plist, B, 0, target.frames, page_seed=None,
                            pack_weights=pack_weights, device=dev)
        self.fuse = [own[n] for n in synth.DRAFT_EXTRA]
        i32 = dict(dtype=torch.int32, device=dev)
        self.tokens = torch.zeros(B, **i32)
        self.sess.in_rows = torch.zeros(B, cfg.d_model, dtype=torch.float32, device=dev)
        self.sess.cross_window = torch.zeros(B, 2, **i32)
        self.ws = torch.empty(ad.draft_input_workspace_size(target.model, B), dtype=torch.uint8,
                              device=dev)
        self.sess.prepare([np.zeros(1, np.int64)] * B)
        self.sess.step_struct.tokens = self.tokens.data_ptr()

    def prefill_encoder(self, encs):
        """The draft's own cross-attention keys / values of the encoder states."""
        self.sess.prefill_encoder(encs)

    def _input(self, first: bool):
        t, s = self.target, self.sess
        if first:
            ad.draft_input(t.model, *self.fuse, self.B, t.out_taps, t.out_hidden, t.cur_layout,
                           t.k_max, t.cu_rows, t.accept_len, t.rows, None, t.out_tokens,
                           t.k_max + 1, t.accept_len, t.out_anchor, s.enc_len, HALF_WINDOW,
                           s.cross_window, s.in_rows, self.ws)
        else:
            ad.draft_input(t.model, *self.fuse, self.B, None, None, t.cur_layout, t.k_max,
                           None, None, t.rows, s.out_hidden, s.out_greedy, 1, None, None, None,
                           0, None, s.in_rows, self.ws)

    def round(self, K: int, out=None):
        """K draft steps after the target step last run; returns a device [B, K] int32
        tensor of drafts (the tokens fed are the pending token, then each draft)."""
        s = self.sess
        out = torch.empty(self.B, K, dtype=torch.int32, device=s.device) if out is None else out
        s.kv_len.zero_()
        # the step's token ids are only validated and scanned (k = 0): its input is in_rows,
        # built by ad_draft_input from the real tokens (the pending token, then each draft)
        self.tokens.zero_()
        for j in range(K):
            self._input(first=j == 0)
            s.run()
            s.commit()
            out[:, j].copy_(s.out_greedy[: self.B])
            self.tokens.copy_(s.out_greedy[: self.B])
        return out


def decode_with_draft(target, runner: DraftRunner, t0, K: int, n_tokens: int, anchor_layer: int):
    """Greedy speculative decode with the audio-conditioned draft: every round verifies
    [pending, d_1..d_k] on the target (with the anchor readout and the draft's taps),
    commits, and drafts the next block.  Round 0 verifies the pending token alone.
    Returns (tokens [B][n_tokens], accepts, drafts, rounds)."""
    B = target.B
    L = target.cfg.n_layers
    target.anchor_layer = anchor_layer
    target.tap_layers = tuple(max(0, L * i // 4 - 1) for i in (1, 2, 3))
    target.out_taps = torch.empty(3, target.max_rows, target.cfg.d_model, dtype=torch.float32,
                                  device=target.device)
    toks = [[] for _ in range(B)]
    accepts, drafts = [], []
    n = target.kv_len.cpu().numpy().astype(np.int64)
    blocks = [np.array([int(t0[b])], np.int64) for b in range(B)]
    rounds = 0
    while min(len(t) for t in toks) < n_tokens:
        drafts.append([blk[1:].copy() for blk in blocks])
        target.step(blocks)
        target.commit()
        nxt = runner.round(K).cpu().numpy()
        res = target.results(keys=("accept_len", "out_tokens", "err"))
        assert res["err"] == 0, f"device error flag {res['err']}"
        a = res["accept_len"]
        accepts.append(a.copy())
        for b in range(B):
            emitted = [int(x) for x in res["out_tokens"][b][: a[b] + 1]]
            toks[b] += emitted
            n[b] += a[b] + 1
            k = _clamp_k(K, int(n[b]))
            blocks[b] = np.concatenate([[emitted[-1]], nxt[b][:k]]).astype(np.int64)
        rounds += 1
    return [t[:n_tokens] for t in toks], accepts, drafts, rounds
