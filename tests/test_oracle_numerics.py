"""Pins of the oracle's storage rounding and extreme-value classes.

Pins: torch's float32 -> bfloat16 conversion (an independent library
routine, round-to-nearest-even), hand-derived bfloat16 values of the
paper's thresholds (Sec. 4.2 constants), and a double-rounding case worked
out by hand.
"""
import numpy as np
import pytest
import torch

from oracle.numerics import round_to, stored_threshold, classify


def _torch_bf16(x32):
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy().astype(np.float64)


def test_bf16_matches_torch_on_random_float32():
    rng = np.random.default_rng(7)
    parts = [
        rng.standard_normal(20000),
        rng.standard_normal(20000) * 1e30,
        rng.standard_normal(20000) * 1e-30,
        np.ldexp(rng.uniform(1, 2, 5000), rng.integers(-140, 127, 5000)),
    ]
    x32 = np.concatenate(parts).astype(np.float32)
    # exact bf16 ties: 1 + 2^-8 style half-way points at many scales
    ties = np.ldexp(1.0 + np.arange(0, 128) / 128.0 + 2.0 ** -8, 3).astype(np.float32)
    x32 = np.concatenate([x32, ties, -ties, np.float32([0.0, -0.0, np.inf, -np.inf])])
    ours = round_to(x32.astype(np.float64), "bf16")
    ref = _torch_bf16(x32)
    assert np.array_equal(ours, ref)


def test_bf16_nan_and_overflow():
    assert np.isnan(round_to(np.array([np.nan]), "bf16")[0])
    # the largest finite bfloat16 is (2 - 2^-7) * 2^127; half an ulp above it
    # rounds to infinity, just below stays finite
    big = np.ldexp(255.0, 120)
    assert round_to(np.array([big]), "bf16")[0] == big
    assert np.isinf(round_to(np.array([big + np.ldexp(1.0, 119)]), "bf16")[0])
    assert round_to(np.array([big + np.ldexp(1.0, 118)]), "bf16")[0] == big


def test_bf16_rounds_directly_from_float64():
    # 1 + 2^-8 is exactly half-way between bf16 neighbours 1 and 1 + 2^-7.
    # A tiny excess makes the nearest bf16 1 + 2^-7; rounding through float32
    # first would lose the excess and tie to even (1.0).
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert round_to(np.array([x]), "bf16")[0] == 1.0 + 2.0 ** -7
    assert round_to(np.array([1.0 + 2.0 ** -8]), "bf16")[0] == 1.0


def test_bf16_subnormal_spacing():
    step = 2.0 ** -133
    x = np.array([3.4 * step, 2.5 * step, -1.5 * step])
    assert np.array_equal(round_to(x, "bf16"), np.array([3.0, 2.0, -2.0]) * step)


def test_thresholds_as_stored():
    # 1e10 = 1.16415... * 2^33; 8 significant bits: round(1.16415*128) = 149
    assert stored_threshold(1e10, "bf16") == 149 * 2.0 ** 26 == 9999220736.0
    # 1e5 = 1.52587... * 2^16 -> 195 * 2^9
    assert stored_threshold(1e5, "bf16") == 195 * 2.0 ** 9 == 99840.0
    # 1e6 = 1.90734... * 2^19 -> 244 * 2^12
    assert stored_threshold(1e6, "bf16") == 244 * 2.0 ** 12 == 999424.0
    assert stored_threshold(1e10, "f32") == 1e10
    assert abs(stored_threshold(1e30, "bf16") / 1e30 - 1) < 2.0 ** -8


def test_classify():
    tn = stored_threshold(1e10, "bf16")
    assert classify(np.nan, tn) == "NAN"
    assert classify(-np.inf, tn) == "INF"
    assert classify(float(round_to(np.array([-1e10]), "bf16")[0]), tn) == "NEAR_INF"
    assert classify(1e30, tn) == "NEAR_INF"
    assert classify(1e6, tn) == "NUMERIC"
    assert classify(0.0, tn) == "NUMERIC"
