"""Greedy verification rule (test infrastructure only).

Paper, section 3 "Speculative Loop": the target scores the drafted block in one pass and
keeps the longest prefix of drafts that matches its own greedy output; a round with L
accepted drafts advances 1 + L tokens (appendix "Cost derivation"), the extra token being
the target's own choice at the first position that was not accepted.
"""
from __future__ import annotations

import numpy as np


def argmax_lowest(v: np.ndarray) -> int:
    """Index of the maximum; among equal maxima the lowest index."""
    v = np.asarray(v)
    m = v.max()
    return int(np.flatnonzero(v == m)[0])


def top2_margin(v: np.ndarray) -> float:
    """Largest value minus the second largest (0 when the maximum is tied)."""
    v = np.asarray(v, dtype=np.float64)
    i = argmax_lowest(v)
    rest = np.delete(v, i)
    return float(v[i] - rest.max())


def accept_length(drafts, greedy) -> int:
    """Longest prefix of drafts d_1..d_k equal to the greedy outputs g_0..g_{k-1}.

    ``greedy[i]`` is the target's argmax at block row i, i.e. its prediction for the
    position of draft d_{i+1}.
    """
    a = 0
    while a < len(drafts) and int(drafts[a]) == int(greedy[a]):
        a += 1
    return a


def emitted_tokens(greedy, a: int):
    """Tokens a verify round outputs: g_0..g_a (a accepted drafts plus the target's token)."""
    return [int(t) for t in greedy[: a + 1]]


def committed_length(n: int, a: int) -> int:
    """KV length after the round: the pending token and the a accepted drafts are kept."""
    return n + a + 1
