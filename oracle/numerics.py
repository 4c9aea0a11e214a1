"""Storage rounding used by the oracle (test infrastructure only).

The decoder computes in float64; values are rounded only where the method stores them
in a narrower format (the KV caches).  bf16 keeps 8 significant bits and float32's
exponent range; rounding is to nearest, ties to even, applied directly to the float64
value (no intermediate float32 step, which could round twice).
"""
from __future__ import annotations

import numpy as np

_DROP = 52 - 7                      # float64 fraction bits removed to keep bf16's 7
_HALF = np.uint64(1 << (_DROP - 1))
_MASK = np.uint64((1 << _DROP) - 1)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value of each float64 element (ties to even), as float64.

    Valid for finite values that are zero or at least 2**-126 in magnitude (bf16 normal
    range); results that overflow bf16 become +/-inf as in IEEE rounding.
    """
    x = np.asarray(x, dtype=np.float64)
    tiny = (x != 0) & (np.abs(x) < 2.0 ** -126)
    if np.any(tiny):
        raise ValueError("round_bf16: subnormal bf16 range is outside the oracle's scope")
    u = x.view(np.uint64) if x.flags.c_contiguous else np.ascontiguousarray(x).view(np.uint64)
    lsb = (u >> np.uint64(_DROP)) & np.uint64(1)
    r = (u + (_HALF - np.uint64(1)) + lsb) & ~_MASK
    out = r.view(np.float64).reshape(x.shape)
    big = np.abs(out) >= 2.0 ** 128
    if np.any(big):
        out = np.where(big, np.copysign(np.inf, x), out)
    return out


def round_f32(x: np.ndarray) -> np.ndarray:
    """Nearest float32 value (IEEE round to nearest even), as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the storage format: 'bf16', 'f32', or 'f64' (no rounding)."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(f"unknown storage dtype {dtype!r}")
