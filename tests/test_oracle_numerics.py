"""Pins for the oracle's storage rounding (CPU only).

bf16 rounding is checked against torch's float32 -> bfloat16 conversion (an independent
library routine, round to nearest even) and against hand-built tie cases.
"""
import numpy as np
import pytest
import torch

from oracle.numerics import round_bf16, round_f32, store
from paper_2608_12703_amd import synth


def test_bf16_matches_torch_on_float32_inputs():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(200000) * s for s in (1e-3, 1.0, 7.0, 1e4)])
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), ref)


def test_bf16_ties_go_to_even():
    one = 1.0
    ulp = 2.0 ** -7                     # bf16 spacing in [1, 2)
    assert round_bf16(np.array([one + ulp / 2]))[0] == one              # tie, even below
    assert round_bf16(np.array([one + 1.5 * ulp]))[0] == one + 2 * ulp  # tie, even above
    assert round_bf16(np.array([one + ulp / 2 + 1e-12]))[0] == one + ulp
    assert round_bf16(np.array([-(one + ulp / 2)]))[0] == -one


def test_bf16_no_double_rounding():
    # 1 + 2^-8 + 2^-30: float32 would round it to the tie 1 + 2^-8 (-> 1.0 in bf16),
    # the exact value is above the tie and must round up.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert round_bf16(np.array([x]))[0] == 1.0 + 2.0 ** -7


def test_bf16_idempotent_and_generator_agrees():
    g = np.random.default_rng(1)
    x = g.standard_normal(10000).astype(np.float32)
    b = synth.to_bf16(x).astype(np.float64)
    np.testing.assert_array_equal(round_bf16(b), b)
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), b)


def test_bf16_overflow_and_subnormal_guard():
    assert np.isinf(round_bf16(np.array([3.5e38]))[0])
    with pytest.raises(ValueError):
        round_bf16(np.array([1e-40]))


def test_f32_and_store():
    x = np.array([1.0 + 2.0 ** -30, 0.1])
    np.testing.assert_array_equal(round_f32(x), np.array([1.0, np.float32(0.1)], np.float64))
    np.testing.assert_array_equal(store(x, "f64"), x)
    with pytest.raises(ValueError):
        store(x, "fp8")
