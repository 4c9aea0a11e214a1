"""Acceptance measures (test infrastructure only).

Paper, section 3 "Speculative Loop" and appendix "Acceptance measures": s_k is the
fraction of rounds whose first k proposals are all accepted (s_0 = 1), conditional
acceptance is a_k^c = s_k / s_{k-1}, restart acceptance is a_1 = s_1, and the mean
number of accepted drafts per round is L = sum_{k=1..K} s_k.  The two-step length
reported beside a_1 and a_2^c is a_1 (1 + a_2^c) (appendix, AnchorDraft results table).
"""
from __future__ import annotations

import numpy as np


def survival(accepted, K: int) -> np.ndarray:
    """s_0..s_K from per-round accepted-draft counts."""
    a = np.asarray(accepted)
    return np.array([np.mean(a >= k) for k in range(K + 1)], dtype=np.float64)


def conditional_acceptance(s: np.ndarray) -> np.ndarray:
    """a_1^c..a_K^c (nan where s_{k-1} = 0)."""
    s = np.asarray(s, np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        return s[1:] / s[:-1]


def mean_accepted_length(s: np.ndarray) -> float:
    return float(np.sum(np.asarray(s, np.float64)[1:]))


def two_step_length(a1: float, a2c: float) -> float:
    return float(a1 * (1.0 + a2c))


def tokens_per_round(accepted) -> float:
    """Output tokens per round: accepted drafts plus the target's own token."""
    return float(np.mean(np.asarray(accepted)) + 1.0)
