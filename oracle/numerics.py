"""Storage rounding and extreme-value classes (oracle; test infrastructure).

Sec. 2.2 of the paper names three extreme-value classes produced by bit
flips: INF, NaN and near-INF, the last defined only by a threshold that
depends on the computation. A value is near-INF here when it is finite and
its magnitude is at least T_near-INF as stored in the storage dtype (the
threshold itself rounded to that dtype, so bf16(1e10) = 9999220736 counts).
"""
from __future__ import annotations

import numpy as np

KINDS = ("NUMERIC", "NEAR_INF", "INF", "NAN")


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), directly
    from float64 (no intermediate float32 rounding). bfloat16 carries 8
    significant bits with float32's exponent range; below 2**-126 the
    spacing is the fixed subnormal step 2**-133. Results beyond the largest
    finite bfloat16 become +-inf; NaN maps to the canonical quiet NaN."""
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, dtype=np.float64, copy=True)
    fin = np.isfinite(x) & (x != 0)
    xf = x[fin]
    _, e = np.frexp(xf)                      # xf = m * 2**e, 0.5 <= |m| < 1
    spacing_exp = np.maximum(e, -125) - 8    # log2 of the unit in the last place
    q = np.ldexp(np.rint(np.ldexp(xf, -spacing_exp)), spacing_exp)
    max_bf16 = np.ldexp(255.0, 120)          # 0x7F7F = (2 - 2**-7) * 2**127
    q = np.where(np.abs(q) > max_bf16, np.copysign(np.inf, q), q)
    out[fin] = q
    out[np.isnan(x)] = np.nan
    return out


def round_to(x, dtype: str) -> np.ndarray:
    """Round to the storage dtype ("bf16", "f32" or "f64"), returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f64":
        return np.array(x, copy=True)
    if dtype == "f32":
        with np.errstate(over="ignore"):
            return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return _round_bf16(x)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def flip_exponent_msb(x: float, dtype: str) -> float:
    """The fault injector's bit flip (Sec. 5.1): the most significant bit of
    the exponent field of the value as stored in dtype (bf16: bit 14 of
    the 16-bit word, f32: bit 30, f64: bit 62). x must already be rounded
    to dtype."""
    if dtype == "f64":
        u = np.array([x], dtype=np.float64).view(np.uint64)
        return float((u ^ np.uint64(1 << 62)).view(np.float64)[0])
    u = np.array([x], dtype=np.float32).view(np.uint32)
    bit = np.uint32(1 << 30)  # bf16 keeps the upper half of the f32 word: its bit 14
    return float((u ^ bit).view(np.float32)[0])


def stored_threshold(t: float, dtype: str) -> float:
    """A threshold as the storage dtype represents it (Sec. 4.2 constants
    compare against stored values)."""
    return float(round_to(np.array([t]), dtype)[0])


def classify(value: float, t_near_inf_stored: float) -> str:
    """Extreme-value class of one stored value (Sec. 2.2)."""
    if np.isnan(value):
        return "NAN"
    if np.isinf(value):
        return "INF"
    if abs(value) >= t_near_inf_stored:
        return "NEAR_INF"
    return "NUMERIC"
