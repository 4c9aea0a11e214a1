"""Pins for the acceptance measures (CPU only)."""
import os

import numpy as np

from oracle.metrics import (conditional_acceptance, mean_accepted_length, survival,
                            tokens_per_round, two_step_length)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "two_step_length.txt")


def test_two_step_length_reproduces_paper_table():
    rows = [ln.split() for ln in open(GOLDEN) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 10
    for _, _, _, a1, a2c, printed in rows:
        assert abs(two_step_length(float(a1), float(a2c)) - float(printed)) <= 0.0015


def test_survival_identities():
    g = np.random.default_rng(0)
    K = 6
    acc = np.minimum(g.geometric(0.25, size=20000) - 1, K)
    s = survival(acc, K)
    assert s[0] == 1.0 and np.all(np.diff(s) <= 0)
    # L = sum_k P(a >= k) = E[a]
    assert abs(mean_accepted_length(s) - acc.mean()) < 1e-12
    # s_k = prod_{j<=k} a_j^c
    np.testing.assert_allclose(np.cumprod(conditional_acceptance(s)), s[1:], rtol=1e-12)
    # geometric agreement: every conditional acceptance is 1 - p
    np.testing.assert_allclose(conditional_acceptance(s)[:4], 0.75, atol=0.02)
    # two-step length = s_1 + s_2
    c = conditional_acceptance(s)
    assert abs(two_step_length(c[0], c[1]) - (s[1] + s[2])) < 1e-12
    assert abs(tokens_per_round(acc) - (1 + acc.mean())) < 1e-12
