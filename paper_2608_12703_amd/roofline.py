"""Algorithmic byte and flop counts of the verify step (what the method must move).

Per step, with s bytes per stored element:
  weights   (L (6 d^2 + 2 d F) + V d) s   self QKV + O, cross Q + O, FFN, tied LM head
                                            (the encoder K/V projections are prefilled)
  cross K/V sum_b 2 L T_b d s              every layer reads every frame's key and value
  self K/V  sum_b 2 L n_b d s              the committed cache
  KV write  sum_b 2 L (k_b + 1) d s        the block's keys and values
Activations (float32 rows, < 1% at the large shapes) are counted per kernel below.
"""
from __future__ import annotations

import hashlib
import os

import numpy as np

HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
BF16_MFMA_PEAK = 2.5e15    # dense bf16 MFMA, flop/s


def elem_bytes(cfg) -> int:
    return 2 if cfg.dtype == "bf16" else 4


def step_bytes(cfg, n, T, k) -> dict:
    s, L, d, F, V = elem_bytes(cfg), cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab
    n, T, k = (np.asarray(x, np.int64) for x in (n, T, k))
    out = {
        "weights": (L * (6 * d * d + 2 * d * F) + V * d) * s,
        "cross_kv": int(np.sum(2 * L * T * d * s)),
        "self_kv": int(np.sum(2 * L * n * d * s)),
        "kv_write": int(np.sum(2 * L * (k + 1) * d * s)),
    }
    out["total"] = sum(out.values())
    return out


def cross_attn_launch_bytes(cfg, T, rows: int) -> int:
    """One layer's cross-attention launch: every frame's K and V of every head, plus the
    float32 query rows read and output rows written."""
    s, d = elem_bytes(cfg), cfg.d_model
    return int(np.sum(2 * np.asarray(T, np.int64) * d * s)) + 2 * rows * d * 4


def step_flops(cfg, n, T, k) -> dict:
    L, d, F, V = cfg.n_layers, cfg.d_model, cfg.d_ffn, cfg.vocab
    n, T, k = (np.asarray(x, np.int64) for x in (n, T, k))
    M = int(np.sum(k + 1))
    return {"gemm": 2 * (L * (6 * d * d + 2 * d * F) + V * d) * M,
            "attention": int(np.sum(4 * (k + 1) * (T + n + k + 1) * d * L))}


# Sources the cross-attention kernel is built from (its file, the shared device helpers
# and the declaration of its argument struct); HBM counter figures taken for one version
# of them are reported only while they are unchanged.
_CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
KERNEL_SOURCES = ("mfma_attn.hip", "common.h")
ARGS_DECL = ("launch.h", "struct AttnArgs {")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(_CSRC, name), "rb") as fh:
            h.update(fh.read())
    name, start = ARGS_DECL
    with open(os.path.join(_CSRC, name)) as fh:
        text = fh.read()
    i = text.index(start)
    h.update(text[i: text.index("};", i) + 2].encode())
    return h.hexdigest()
