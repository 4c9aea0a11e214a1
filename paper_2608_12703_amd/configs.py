"""Workload presets for the batched speculative-verify step.

Every preset is a Whisper-shape pre-LN decoder (64-wide heads, 448 positions, up to
1500 encoder frames).  The paper verifies a drafted block in one decoder pass and keeps
the longest greedy-matching prefix (section 3, "Speculative Loop"); it names
Whisper-large-v3 as one of its targets (appendix "Whisper Cross-Architecture Check"),
which fixes the large shapes below.  Acceptance is planted: drafts agree with the
target's greedy continuation for a Geometric(p) number of positions, which gives the
restart acceptance 1-p that the paper measures in the 0.6-0.76 range (section 4,
"Restart and Continuation").
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

HEAD_DIM = 64          # per-head width of every attention layer
MAX_POS = 448          # decoder positions (learned position table rows)
MAX_FRAMES = 1500      # encoder frames after the convolutional stride
SOT_TOKEN = 50258      # start-of-transcript id used to open a decode at position 0
PAGE = 16              # tokens per self-KV page (one 16-key attention tile)


@dataclass(frozen=True)
class Config:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int
    dtype: str                  # "f32" or "bf16" storage of weights / encoder / KV
    batch: int
    k: int                      # draft length (max draft length for ragged batches)
    k_min: int = -1             # ragged: k_b ~ U{k_min..k}; -1 -> fixed k
    frames: int = MAX_FRAMES    # encoder frames (max for ragged batches)
    frames_min: int = -1        # ragged: T_b ~ U{frames_min..frames}; -1 -> fixed
    kv_max: int = 0             # committed prefix length n_b ~ U{0..kv_max} (clamped per k_b)
    geo_p: float = 0.0          # planted agreement: G ~ Geometric(p) on {0,1,2,...}
    decode_tokens: int = 0      # loop configs: tokens to decode
    draft_heads: int = 0        # linear draft heads on the final hidden state
    anchor_lambda: float = 0.0  # drift stress: Poisson gap between misalignment anchors
    max_pos: int = MAX_POS      # decoder positions (rows of the learned position table)
    seed: int = 0
    notes: str = ""

    @property
    def head_dim(self) -> int:
        return HEAD_DIM

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)

    def n_params(self) -> int:
        d, F, L, V = self.d_model, self.d_ffn, self.n_layers, self.vocab
        per_layer = 3 * d * d + 3 * d + d * d + d + d * d + d + 2 * d * d + 2 * d \
            + d * d + d + F * d + F + d * F + d + 6 * d
        return L * per_layer + V * d + self.max_pos * d + 2 * d


TINY_FP32 = Config(
    name="tiny_fp32", n_layers=4, d_model=384, n_heads=6, d_ffn=1536, vocab=51865,
    dtype="f32", batch=1, k=4, decode_tokens=64, draft_heads=4,
    notes="64-token greedy decode from position 0; drafts from 4 linear heads")

SMALL_BF16 = Config(
    name="small_bf16", n_layers=12, d_model=768, n_heads=12, d_ffn=3072, vocab=51865,
    dtype="bf16", batch=16, k=4, kv_max=224, geo_p=0.3)

LARGE_V3_BF16 = Config(
    name="large_v3_bf16", n_layers=32, d_model=1280, n_heads=20, d_ffn=5120, vocab=51866,
    dtype="bf16", batch=32, k=6, kv_max=MAX_POS - 1 - 6, geo_p=0.25)

RAGGED_LARGE_V3 = Config(
    name="ragged_large_v3", n_layers=32, d_model=1280, n_heads=20, d_ffn=5120, vocab=51866,
    dtype="bf16", batch=64, k=8, k_min=2, frames=1500, frames_min=200,
    kv_max=MAX_POS - 1, geo_p=0.2)

DRIFT_STRESS = Config(
    name="drift_stress", n_layers=32, d_model=1280, n_heads=20, d_ffn=5120, vocab=51866,
    dtype="bf16", batch=32, k=8, decode_tokens=MAX_POS, anchor_lambda=40.0)

CONFIGS = {c.name: c for c in (TINY_FP32, SMALL_BF16, LARGE_V3_BF16, RAGGED_LARGE_V3,
                               DRIFT_STRESS)}
