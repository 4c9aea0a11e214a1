"""Float64 Whisper-shape decoder, one-pass verification and greedy decoding.

TEST INFRASTRUCTURE ONLY (see the package header).  Written to be read against the
paper, not to be fast.

The method (paper, section 3 "Speculative Loop"): the target checks a drafted block in
one pass and keeps the longest prefix that matches its own greedy output; under exact
arithmetic this returns the target-greedy sequence.  The accepted tokens and their
cached states feed the next round (appendix "Real cached loop").

The paper defines no decoder; its Whisper-large-v3 target fixes the shape used here: a
pre-LN decoder with learned positions, per layer
  x <- x + SelfAttn(LN1(x))   (causal, over the KV cache and the block)
  x <- x + CrossAttn(LN2(x))  (over the encoder's projected states)
  x <- x + W2 GELU(W1 LN3(x) + b1) + b2
then LN_f and a head tied to the token embedding.  Heads are 64 wide with score scale
1/8; LayerNorm uses the biased variance and eps = 1e-5; GELU is the exact erf form.

Precision: everything is float64 except where the method stores values: keys and
values written to the caches are rounded to the cache's storage format, and the argmax
is taken on logits rounded to float32, the precision in which the GPU path decides it.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
from scipy.special import erf

from .accept import accept_length, argmax_lowest, emitted_tokens, top2_margin
from .numerics import round_f32, store

HEAD = 64
EPS = 1e-5
MAX_POS = 448   # rows of the Whisper-shape position table (a model may carry another)


# ---------------------------------------------------------------------- sublayers

def layer_norm(x, g, b):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + EPS) * g + b


def gelu(u):
    return 0.5 * u * (1.0 + erf(u / np.sqrt(2.0)))


def softmax(s):
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, K, V, visible):
    """Multi-head attention for a few query rows.

    q: [r, H, 64]; K, V: [n_keys, H, 64]; row i sees keys 0..visible[i]-1, or, when
    visible[i] is a boolean array over the keys, the keys it marks.
    Returns [r, H, 64].
    """
    out = np.empty_like(q)
    for i in range(q.shape[0]):
        sel = np.arange(int(visible[i])) if np.ndim(visible[i]) == 0 else np.flatnonzero(visible[i])
        s = np.einsum("hd,thd->ht", q[i], K[sel]) / np.sqrt(HEAD)
        out[i] = np.einsum("ht,thd->hd", softmax(s), V[sel])
    return out


def attention_probs(q, K, visible):
    """Attention weights of a few query rows, per head: [r, H, n_keys], the softmax of
    q.k / 8 over keys 0..visible[i]-1 (zero past them)."""
    P = np.zeros((q.shape[0], q.shape[1], K.shape[0]))
    for i in range(q.shape[0]):
        nv = int(visible[i])
        s = np.einsum("hd,thd->ht", q[i], K[:nv]) / np.sqrt(HEAD)
        P[i, :, :nv] = softmax(s)
    return P


# ---------------------------------------------------------------------- model / state

class Model:
    """Parameters (float32 arrays from the generator) and the cache storage format.

    ``kv_dtype`` is 'bf16', 'f32' or 'f64'; it defaults to the model's storage dtype.
    """

    def __init__(self, cfg, params: dict, kv_dtype: str | None = None):
        self.L, self.d, self.H = cfg.n_layers, cfg.d_model, cfg.n_heads
        self.F, self.V = cfg.d_ffn, cfg.vocab
        self.params = params
        self.kv_dtype = kv_dtype or cfg.dtype
        # decoder positions: the rows of the learned position table
        self.max_pos = len(params["pos_emb"])

    def w(self, name):
        return np.asarray(self.params[name], dtype=np.float64)

    def lw(self, layer, name):
        return self.w(f"l{layer}.{name}")


@dataclass
class SeqState:
    """One sequence: committed self-KV, encoder K/V, pending token.

    self_kv[l] = (K, V), each [n, H, 64] holding stored (rounded) values.
    cross[l]   = (K, V), each [T, H, 64].
    t0         = the last emitted token, not yet fed (it sits at position n).
    """
    self_kv: list
    cross: list
    t0: int

    @property
    def n(self) -> int:
        return int(self.self_kv[0][0].shape[0])


def cross_kv(model: Model, enc: np.ndarray):
    """Encoder keys/values per layer: K = enc W_k^T, V = enc W_v^T + b_v (stored)."""
    enc = np.asarray(enc, dtype=np.float64)
    T, d, H = enc.shape[0], model.d, model.H
    out = []
    for layer in range(model.L):
        kv = enc @ model.lw(layer, "w_xkv").T + model.lw(layer, "b_xkv")
        K = store(kv[:, :d], model.kv_dtype).reshape(T, H, HEAD)
        V = store(kv[:, d:], model.kv_dtype).reshape(T, H, HEAD)
        out.append((K, V))
    return out


def new_state(model: Model, cross, t0: int, prefix_kv=None) -> SeqState:
    """State with an optional committed prefix; prefix_kv is [L, 2, n, H, 64]."""
    kv = []
    for layer in range(model.L):
        if prefix_kv is None:
            z = np.zeros((0, model.H, HEAD))
            kv.append((z, z.copy()))
        else:
            kv.append((np.asarray(prefix_kv[layer, 0], np.float64),
                       np.asarray(prefix_kv[layer, 1], np.float64)))
    return SeqState(kv, cross, int(t0))


@dataclass
class BlockOut:
    logits: np.ndarray      # [r, V] float64
    hidden: np.ndarray      # [r, d] final-LN output
    new_kv: list            # per layer (K, V) of the block rows, [r, H, 64], stored
    xattn: np.ndarray | None = None   # [r, H, T] cross-attention weights at the probed layer
    taps: np.ndarray | None = None    # [n_taps, r, d] residual stream after the tapped layers


def tree_depths(parents):
    """Depth of every node of a draft tree (node 0, the root, has depth 0; parent[i] < i)."""
    depth = [0] * len(parents)
    for i in range(1, len(parents)):
        depth[i] = depth[int(parents[i])] + 1
    return depth


def tree_visibility(parents, n: int):
    """Keys each block row may attend to in a tree block: the n committed positions and
    the row's ancestors and itself ([r, n + r] booleans)."""
    r = len(parents)
    vis = np.zeros((r, n + r), dtype=bool)
    vis[:, :n] = True
    for i in range(r):
        j = i
        while True:
            vis[i, n + j] = True
            if j == 0:
                break
            j = int(parents[j])
    return vis


def forward_block(model: Model, state: SeqState, tokens, probe_layer: int | None = None,
                  in_rows=None, cross_window=None, taps=None, parents=None) -> BlockOut:
    """One causal decoder pass over ``tokens`` placed at positions n..n+r-1.  With
    ``probe_layer`` set, also returns that layer's cross-attention weights.

    in_rows [r, d]: replaces the token embedding of the rows (the position embedding is
    still added).  cross_window (lo, hi): the rows attend to frames lo..hi-1 only.
    taps: list of layer indices; the residual stream after each is returned in
    ``BlockOut.taps`` [len(taps), r, d].
    parents: a draft tree over the rows (parents[0] ignored, parents[i] < i): row i
    sits at position n + depth(i) and attends to the committed keys and its ancestors."""
    tokens = np.asarray(tokens, dtype=np.int64)
    r, n, d, H = len(tokens), state.n, model.d, model.H
    if n + r > model.max_pos:
        raise ValueError("block runs past the last decoder position")
    pos = n + (np.arange(r) if parents is None else np.asarray(tree_depths(parents)))
    self_vis = pos + 1 if parents is None else tree_visibility(parents, n)
    emb = model.w("tok_emb")[tokens] if in_rows is None else np.asarray(in_rows, np.float64)
    x = emb + model.w("pos_emb")[pos]
    tapped = {}
    new_kv = []
    xattn = None
    for layer in range(model.L):
        h = layer_norm(x, model.lw(layer, "ln1_g"), model.lw(layer, "ln1_b"))
        qkv = h @ model.lw(layer, "w_qkv").T + model.lw(layer, "b_qkv")
        q = qkv[:, :d].reshape(r, H, HEAD)
        k = store(qkv[:, d:2 * d], model.kv_dtype).reshape(r, H, HEAD)
        v = store(qkv[:, 2 * d:], model.kv_dtype).reshape(r, H, HEAD)
        K = np.concatenate([state.self_kv[layer][0], k])
        V = np.concatenate([state.self_kv[layer][1], v])
        a = attention(q, K, V, visible=self_vis).reshape(r, d)
        x = x + a @ model.lw(layer, "w_o").T + model.lw(layer, "b_o")

        h = layer_norm(x, model.lw(layer, "ln2_g"), model.lw(layer, "ln2_b"))
        q = (h @ model.lw(layer, "w_xq").T + model.lw(layer, "b_xq")).reshape(r, H, HEAD)
        Kx, Vx = state.cross[layer]
        if cross_window is not None:
            Kx, Vx = Kx[cross_window[0]: cross_window[1]], Vx[cross_window[0]: cross_window[1]]
        a = attention(q, Kx, Vx, visible=np.full(r, Kx.shape[0])).reshape(r, d)
        if layer == probe_layer:
            xattn = attention_probs(q, Kx, visible=np.full(r, Kx.shape[0]))
        x = x + a @ model.lw(layer, "w_xo").T + model.lw(layer, "b_xo")

        h = layer_norm(x, model.lw(layer, "ln3_g"), model.lw(layer, "ln3_b"))
        u = gelu(h @ model.lw(layer, "w_1").T + model.lw(layer, "b_1"))
        x = x + u @ model.lw(layer, "w_2").T + model.lw(layer, "b_2")
        new_kv.append((k, v))
        tapped[layer] = x.copy()
    hidden = layer_norm(x, model.w("lnf_g"), model.w("lnf_b"))
    logits = hidden @ model.w("tok_emb").T
    tap_out = None if taps is None else np.stack([tapped[t] for t in taps])
    return BlockOut(logits, hidden, new_kv, xattn, tap_out)


# ---------------------------------------------------------------------- verify / AR

@dataclass
class VerifyOut:
    greedy: list          # g_0..g_k: argmax at each block row
    accepted: int         # a: longest greedy-matching draft prefix
    emitted: list         # g_0..g_a
    margins: list         # top-1 minus top-2 of the float32-rounded logits, per row
    logits: np.ndarray    # [k+1, V] float64
    hidden: np.ndarray    # [k+1, d]
    state: SeqState       # state after commit
    block_kv: list        # per layer (K, V) written for all k+1 block rows, [k+1, H, 64]
    taps: np.ndarray | None = None   # residual stream after the requested layers [t, k+1, d]


def decide(logits: np.ndarray):
    """Greedy token and top-2 margin of each row, on float32-rounded logits."""
    dec = round_f32(logits)
    return [argmax_lowest(row) for row in dec], [top2_margin(row) for row in dec]


def commit(state: SeqState, out: BlockOut, a: int, t_next: int) -> SeqState:
    kv = [(np.concatenate([K, k[: a + 1]]), np.concatenate([V, v[: a + 1]]))
          for (K, V), (k, v) in zip(state.self_kv, out.new_kv)]
    return SeqState(kv, state.cross, int(t_next))


def verify(model: Model, state: SeqState, drafts, taps=None) -> VerifyOut:
    """Score [t0, d_1..d_k] in one pass, accept, emit and commit.  ``taps``: layers whose
    output residual stream is also returned (no effect on the result)."""
    drafts = [int(t) for t in drafts]
    out = forward_block(model, state, [state.t0] + drafts, taps=taps)
    greedy, margins = decide(out.logits)
    a = accept_length(drafts, greedy)
    return VerifyOut(greedy, a, emitted_tokens(greedy, a), margins, out.logits, out.hidden,
                     commit(state, out, a, greedy[a]), out.new_kv, out.taps)


def ar_step(model: Model, state: SeqState) -> VerifyOut:
    """One autoregressive greedy step: a verify round with no drafts."""
    return verify(model, state, [])


def ar_decode(model: Model, state: SeqState, n_tokens: int):
    """Plain greedy decoding, one position at a time. Returns (tokens, margins, state)."""
    toks, margins = [], []
    for _ in range(n_tokens):
        r = ar_step(model, state)
        toks.append(r.emitted[0])
        margins.append(r.margins[0])
        state = r.state
    return toks, margins, state


def draft_heads(heads_w: np.ndarray, hidden_row: np.ndarray):
    """Linear draft heads: d_i = argmax(W_i h) on float32-rounded logits, lowest index."""
    h = np.asarray(hidden_row, np.float64)
    return [argmax_lowest(round_f32(np.asarray(W, np.float64) @ h)) for W in heads_w]


def spec_decode_heads(model: Model, state: SeqState, heads_w, n_tokens: int):
    """Speculative greedy decode with linear draft heads.

    Round 0 is an AR step (no hidden state exists yet for the heads); every later round
    drafts with the heads on the final hidden row of the last accepted position, verifies,
    and commits.  The draft length is clamped so the block never passes the last position.
    Returns (emitted tokens truncated to n_tokens, per-round accepted counts, rounds).
    """
    toks, accepts, rounds = [], [], []
    r = ar_step(model, state)
    toks += r.emitted
    hidden, state = r.hidden[r.accepted], r.state
    while len(toks) < n_tokens:
        k = min(len(heads_w), model.max_pos - 1 - state.n)
        drafts = draft_heads(heads_w[:k], hidden)
        r = verify(model, state, drafts)
        rounds.append(r)
        accepts.append(r.accepted)
        toks += r.emitted
        hidden, state = r.hidden[r.accepted], r.state
    return toks[:n_tokens], accepts, rounds


# ---------------------------------------------------------------------- anchor readout

@dataclass
class Anchor:
    frame: int            # argmax over frames of the head-averaged weights (lowest index)
    peak: float           # the head-averaged weight there
    margin: float         # its top-1 minus top-2 over frames
    mean: np.ndarray      # [T] head-averaged weights of the row


def anchor_of(xattn_row: np.ndarray) -> Anchor:
    """Audio position from the target's verification attention (paper, section "Correction
    and Cost", paragraph "Verification-Attention Correction"; appendix "Runtime
    Correction"): average one query row's cross-attention weights over the heads at the
    selected layer and take the peak frame.  xattn_row: [H, T]."""
    mean = np.asarray(xattn_row, np.float64).mean(axis=0)
    t = argmax_lowest(mean)
    return Anchor(t, float(mean[t]), top2_margin(mean) if mean.size > 1 else float("inf"), mean)


def verify_with_anchor(model: Model, state: SeqState, drafts, layer: int, taps=None):
    """verify() plus the anchor read from the cross-attention at ``layer`` of block row a,
    the last verified position (its output is the bonus token, so its audio attention
    marks where the next draft should start)."""
    drafts = [int(t) for t in drafts]
    out = forward_block(model, state, [state.t0] + drafts, probe_layer=layer, taps=taps)
    greedy, margins = decide(out.logits)
    a = accept_length(drafts, greedy)
    res = VerifyOut(greedy, a, emitted_tokens(greedy, a), margins, out.logits, out.hidden,
                    commit(state, out, a, greedy[a]), out.new_kv, out.taps)
    return res, anchor_of(out.xattn[a])


# ---------------------------------------------------------------------- tree verification

@dataclass
class TreeVerifyOut:
    greedy: list          # g at every node
    margins: list
    path: list            # accepted node indices from the root: [0, u_1, .., u_a]
    accepted: int         # a
    emitted: list         # g along the path: a accepted drafts plus the target's token
    state: SeqState       # committed: the path's keys / values at positions n .. n + a


def verify_tree(model: Model, state: SeqState, tokens, parents) -> TreeVerifyOut:
    """Verify a draft tree in one pass (appendix "Tree-decoder implementation check":
    all nodes in one pass with a tree attention mask).  tokens[0] is the pending token
    at the root, tokens[i] the draft of node i with parent parents[i] < i.  From the root,
    the walk moves to the child whose token equals the current node's greedy token (the
    lowest-index such child); the accepted drafts are the nodes passed, the emitted
    tokens the greedy tokens along the path, and the committed cache holds the path."""
    tokens = [int(t) for t in tokens]
    out = forward_block(model, state, tokens, parents=parents)
    greedy, margins = decide(out.logits)
    path = [0]
    while True:
        u = path[-1]
        nxt = [c for c in range(1, len(tokens)) if int(parents[c]) == u and tokens[c] == greedy[u]]
        if not nxt:
            break
        path.append(nxt[0])
    a = len(path) - 1
    kv = [(np.concatenate([K, k[path]]), np.concatenate([V, v[path]]))
          for (K, V), (k, v) in zip(state.self_kv, out.new_kv)]
    return TreeVerifyOut(greedy, margins, path, a, [greedy[u] for u in path],
                         SeqState(kv, state.cross, greedy[path[-1]]))
