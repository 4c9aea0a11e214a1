"""Seeded synthetic inputs for the speculative-verify step.

This module only draws random numbers and arranges them; it holds none of the decoder's
arithmetic.  Both the CPU oracle and the GPU harness take their inputs from here, so the
two sides see the same bytes.

Streams.  Every random quantity comes from ``SeedSequence(seed, spawn_key=(stream, i))``
with a fixed stream id and an index (parameter number or sequence number), so a
sequence's inputs do not depend on the batch it sits in and a subset of sequences can be
regenerated alone.

Distributions (paper-silent points, chosen to match a random-init N(0, 0.02) model):

* matrices, embeddings, biases: N(0, 0.02); LayerNorm gain 1 + N(0, 0.02), shift
  N(0, 0.02).  The key projections carry no bias (their bias segments are zero).
* encoder states: N(0, 1).
* committed self-KV prefix: N(0, (0.02 sqrt(d))^2), the spread a unit-variance
  LayerNorm output times N(0, 0.02) weights gives to the model's own keys and values.
* draft agreement: G ~ Geometric(p) on {0, 1, ...}; drafts copy the greedy continuation
  for G positions, the next draft is a uniform token different from the greedy one, the
  rest are uniform.  Acceptance is then exactly min(G, k) (restart acceptance 1 - p, the
  quantity of section 3, "Speculative Loop").
* drift anchors: gaps ~ Poisson(lambda) (at least 1), offset +1 or -1 by a fair coin.

bf16 storage: values are rounded to the nearest bf16 (ties to even) and kept as float32
arrays whose low 16 bits are zero.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import Config, HEAD_DIM, MAX_POS, SOT_TOKEN

# stream ids (fixed order; never renumber)
S_WEIGHTS, S_ENCODER, S_KVLEN, S_PREFIX, S_GEO, S_FILL, S_ANCHOR, S_HEADS, S_SHAPE, S_DRAFT = range(10)


def _rng(seed: int, stream: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(stream, index))))


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); float32 result."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    x = x.astype(np.float32, copy=False)
    return to_bf16(x) if dtype == "bf16" else x


# --------------------------------------------------------------------------- weights

GLOBAL_PARAMS = ("tok_emb", "pos_emb", "lnf_g", "lnf_b")
LAYER_PARAMS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
                "ln2_g", "ln2_b", "w_xq", "b_xq", "w_xkv", "b_xkv", "w_xo", "b_xo",
                "ln3_g", "ln3_b", "w_1", "b_1", "w_2", "b_2")


def param_specs(cfg: Config):
    """Ordered (name, shape) list; the order is the C-ABI parameter order.

    Matrices are stored [out_features, in_features] row-major.
    """
    d, F, V = cfg.d_model, cfg.d_ffn, cfg.vocab
    shapes = {"tok_emb": (V, d), "pos_emb": (cfg.max_pos, d), "lnf_g": (d,), "lnf_b": (d,),
              "ln1_g": (d,), "ln1_b": (d,), "w_qkv": (3 * d, d), "b_qkv": (3 * d,),
              "w_o": (d, d), "b_o": (d,), "ln2_g": (d,), "ln2_b": (d,),
              "w_xq": (d, d), "b_xq": (d,), "w_xkv": (2 * d, d), "b_xkv": (2 * d,),
              "w_xo": (d, d), "b_xo": (d,), "ln3_g": (d,), "ln3_b": (d,),
              "w_1": (F, d), "b_1": (F,), "w_2": (d, F), "b_2": (d,)}
    out = [(n, shapes[n]) for n in GLOBAL_PARAMS]
    for layer in range(cfg.n_layers):
        out += [(f"l{layer}.{n}", shapes[n]) for n in LAYER_PARAMS]
    return out


def make_param(cfg: Config, index: int, name: str, shape, seed: int | None = None) -> np.ndarray:
    seed = cfg.seed if seed is None else seed
    g = _rng(seed, S_WEIGHTS, index)
    base = name.split(".")[-1]
    x = g.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
    if base.endswith("_g"):
        x += np.float32(1.0)
    d = cfg.d_model
    if base == "b_qkv":
        x[d:2 * d] = 0.0          # no key bias
    if base == "b_xkv":
        x[0:d] = 0.0              # no key bias
    return _store(x, cfg.dtype)


def make_params(cfg: Config, seed: int | None = None) -> dict:
    """All parameters as float32 arrays (bf16-representable for bf16 configs)."""
    return {name: make_param(cfg, i, name, shape, seed)
            for i, (name, shape) in enumerate(param_specs(cfg))}


def make_draft_heads(cfg: Config, seed: int | None = None) -> np.ndarray:
    """Linear draft heads [n_heads, V, d] ~ N(0, 0.02), no bias."""
    seed = cfg.seed if seed is None else seed
    out = np.empty((cfg.draft_heads, cfg.vocab, cfg.d_model), np.float32)
    for i in range(cfg.draft_heads):
        out[i] = _rng(seed, S_HEADS, i).standard_normal((cfg.vocab, cfg.d_model),
                                                         dtype=np.float32) * np.float32(0.02)
    return _store(out, cfg.dtype)


def draft_config(cfg: Config) -> Config:
    """The audio-conditioned draft block of a target: one decoder layer of the target's
    width and heads with a feed-forward width of twice the model width (the paper's
    drafts use 1024/2048 and 2048/4096)."""
    return cfg.with_(name=cfg.name + "_draft", n_layers=1, d_ffn=2 * cfg.d_model)


DRAFT_EXTRA = ("w_fuse", "b_fuse", "w_in", "b_in")


def draft_param_specs(cfg: Config):
    """(name, shape) of the draft's own parameters: the block (layer 0) and its final
    LayerNorm in the C-ABI order of a one-layer model (the token and position tables are
    the target's), then the input projections: w_fuse [d, 4d] maps four target
    representations to one feature, w_in [d, 2d] maps (feature, token embedding) to the
    block's input."""
    dc, d = draft_config(cfg), cfg.d_model
    specs = [(n, sh) for n, sh in param_specs(dc) if n not in ("tok_emb", "pos_emb")]
    return specs + [("w_fuse", (d, 4 * d)), ("b_fuse", (d,)), ("w_in", (d, 2 * d)), ("b_in", (d,))]


def make_draft_params(cfg: Config, seed: int | None = None) -> dict:
    """Random-init draft parameters (N(0, 0.02); LayerNorm gains 1 + N(0, 0.02))."""
    seed = cfg.seed if seed is None else seed
    out = {}
    for i, (name, shape) in enumerate(draft_param_specs(cfg)):
        g = _rng(seed, S_DRAFT, i)
        x = g.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
        if name.split(".")[-1].endswith("_g"):
            x += np.float32(1.0)
        d = cfg.d_model
        if name.split(".")[-1] == "b_qkv":
            x[d: 2 * d] = 0.0                # keys carry no bias, as in the target
        if name.split(".")[-1] == "b_xkv":
            x[:d] = 0.0
        out[name] = _store(x, cfg.dtype)
    return out


# --------------------------------------------------------------------- per-sequence data

def make_encoder(cfg: Config, b: int, frames: int, seed: int | None = None) -> np.ndarray:
    """Encoder states of sequence b: [frames, d] ~ N(0, 1)."""
    seed = cfg.seed if seed is None else seed
    x = _rng(seed, S_ENCODER, b).standard_normal((cfg.frames, cfg.d_model), dtype=np.float32)
    return _store(x[:frames], cfg.dtype)


def make_prefix_kv(cfg: Config, b: int, n: int, seed: int | None = None) -> np.ndarray:
    """Committed self-KV of sequence b: [L, 2(K,V), n, H, 64] ~ N(0, (0.02 sqrt d)^2)."""
    seed = cfg.seed if seed is None else seed
    g = _rng(seed, S_PREFIX, b)
    sigma = np.float32(0.02 * np.sqrt(cfg.d_model))
    x = g.standard_normal((cfg.n_layers, 2, n, cfg.n_heads, HEAD_DIM), dtype=np.float32) * sigma
    return _store(x, cfg.dtype)


@dataclass
class StepWorkload:
    """Shapes and planted-agreement draws of one batched verify step."""
    k: np.ndarray        # [B] draft length per sequence
    n: np.ndarray        # [B] committed KV length per sequence
    T: np.ndarray        # [B] encoder frames per sequence
    t0: np.ndarray       # [B] pending token (fed at position n)
    G: np.ndarray        # [B] planted agreement length
    fill_ne: list        # per seq [k_b] uniform on {0..V-2} (mapped to "not the greedy token")
    fill_any: list       # per seq [k_b] uniform on {0..V-1}

    @property
    def batch(self) -> int:
        return len(self.k)

    @property
    def rows(self) -> int:
        return int(np.sum(self.k + 1))


def make_step_workload(cfg: Config, seed: int | None = None, batch: int | None = None) -> StepWorkload:
    seed = cfg.seed if seed is None else seed
    B = cfg.batch if batch is None else batch
    V = cfg.vocab
    k = np.empty(B, np.int64)
    n = np.empty(B, np.int64)
    T = np.empty(B, np.int64)
    t0 = np.empty(B, np.int64)
    G = np.empty(B, np.int64)
    fill_ne, fill_any = [], []
    for b in range(B):
        gs = _rng(seed, S_SHAPE, b)
        k[b] = cfg.k if cfg.k_min < 0 else gs.integers(cfg.k_min, cfg.k + 1)
        T[b] = cfg.frames if cfg.frames_min < 0 else gs.integers(cfg.frames_min, cfg.frames + 1)
        kv_hi = min(cfg.kv_max, cfg.max_pos - 1 - int(k[b]))
        n[b] = _rng(seed, S_KVLEN, b).integers(0, kv_hi + 1)
        gp = _rng(seed, S_GEO, b)
        G[b] = (gp.geometric(cfg.geo_p) - 1) if cfg.geo_p > 0 else 0
        gf = _rng(seed, S_FILL, b)
        t0[b] = gf.integers(0, V)
        fill_ne.append(gf.integers(0, V - 1, size=int(k[b])))
        fill_any.append(gf.integers(0, V, size=int(k[b])))
    return StepWorkload(k, n, T, t0, G, fill_ne, fill_any)


def plant_drafts(y: np.ndarray, G: int, fill_ne: np.ndarray, fill_any: np.ndarray) -> np.ndarray:
    """Drafts d_1..d_k from the greedy continuation y_1..y_k.

    d_i = y_i for i <= G; d_{G+1} is a token different from y_{G+1}; later drafts are
    uniform.  The longest greedy-matching prefix is then exactly min(G, k).
    """
    k = len(y)
    d = np.empty(k, np.int64)
    for i in range(k):             # i is the 0-based index of draft d_{i+1}
        if i < G:
            d[i] = y[i]
        elif i == G:
            f = int(fill_ne[i])
            d[i] = f + (f >= int(y[i]))
        else:
            d[i] = fill_any[i]
    return d


# ----------------------------------------------------------------------- drift stress

@dataclass
class DriftPlan:
    """Misalignment anchors of one sequence for the drift-stress decode loop."""
    anchors: np.ndarray     # increasing positions in [1, MAX_POS]
    signs: np.ndarray       # +1 / -1 offset applied from each anchor on
    fill_ne: np.ndarray     # [MAX_POS + 2] uniform on {0..V-2}


def make_drift_plan(cfg: Config, b: int, seed: int | None = None) -> DriftPlan:
    seed = cfg.seed if seed is None else seed
    g = _rng(seed, S_ANCHOR, b)
    anchors, signs = [], []
    p = 0
    while True:
        p += max(1, int(g.poisson(cfg.anchor_lambda)))
        if p > MAX_POS:
            break
        anchors.append(p)
        signs.append(1 if g.integers(0, 2) == 1 else -1)
    fill = _rng(seed, S_FILL, b).integers(0, cfg.vocab - 1, size=MAX_POS + 2)
    return DriftPlan(np.asarray(anchors, np.int64), np.asarray(signs, np.int64), fill)


def plant_drift(y: np.ndarray, n: int, k: int, plan: DriftPlan) -> np.ndarray:
    """Drafts for positions n+1..n+k of a sequence whose greedy tokens are y[0..].

    y[j] is the target's greedy token at position j (y[0] is the start token).  Let p be
    the first anchor with p > n.  Drafts before p copy y; from p on they copy y shifted by
    the anchor's offset, and where the shifted token equals y[j] (or falls outside y) a
    token different from y[j] is used, so the round is rejected exactly at p.  Once the
    committed length passes p the next anchor takes over (re-anchoring after verification).
    """
    idx = np.searchsorted(plan.anchors, n, side="right")
    p = int(plan.anchors[idx]) if idx < len(plan.anchors) else MAX_POS + 10
    sgn = int(plan.signs[idx]) if idx < len(plan.anchors) else 0
    d = np.empty(k, np.int64)
    for i in range(k):
        j = n + 1 + i
        if j < p:
            d[i] = y[j]
        else:
            src = j + sgn
            cand = int(y[src]) if 0 <= src < len(y) else -1
            if cand < 0 or cand == int(y[j]):
                f = int(plan.fill_ne[j])
                cand = f + (f >= int(y[j]))
            d[i] = cand
    return d


def decode_start_token() -> int:
    return SOT_TOKEN
