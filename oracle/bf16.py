"""Oracle-side number formats: exact bf16 decoding and single rounding of a
float64 value to bf16 or fp32 (round to nearest, ties to even).

The paper fixes no rounding mode; the codec's reading is that every value is
rounded once, from the exact (float64) result, to the output type.  Rounding
float64 -> float32 -> bf16 would round twice and can differ from a single
rounding, so ``round_bf16`` works from the float64 value directly.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from __future__ import annotations

import numpy as np

# bf16 = 1 sign bit, 8 exponent bits (bias 127), 7 stored fraction bits.
_BF16_SIG_BITS = 8            # significant bits including the implicit one
_BF16_MIN_QUANTUM_EXP = -133  # smallest subnormal 2**-133 = 2**(-126 - 7)
_BF16_OVERFLOW = 2.0 ** 128   # first value past the largest finite bf16


def decode_bf16(bits: np.ndarray, dtype=np.float64) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (or float32; both exact: bf16 is the
    top half of a float32)."""
    b = np.asarray(bits)
    if b.dtype != np.uint16:
        b = b.astype(np.uint16)
    f = (b.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if dtype == np.float32:
        return f
    with np.errstate(invalid="ignore"):
        return f.astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), returned as float64.

    Overflow gives +-inf, NaN stays NaN, the sign of zero is kept.
    """
    x = np.asarray(x, dtype=np.float64)
    out = x.copy()
    fin = np.isfinite(x)
    xf = x[fin]
    _, e = np.frexp(xf)                       # xf = m * 2**e, 0.5 <= |m| < 1
    qexp = np.maximum(e - _BF16_SIG_BITS, _BF16_MIN_QUANTUM_EXP)
    r = np.ldexp(np.round(np.ldexp(xf, -qexp)), qexp)   # np.round: ties to even
    big = np.abs(r) >= _BF16_OVERFLOW
    r[big] = np.copysign(np.inf, xf[big])
    out[fin] = r
    return out


def encode_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> uint16 bf16 bit patterns with one round-to-nearest-even step."""
    r = round_bf16(x)
    bits = (r.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    bits[np.isnan(r)] = np.uint16(0x7FC0)
    return bits


def round_f32(x: np.ndarray) -> np.ndarray:
    """Round float64 values to float32 (IEEE conversion, ties to even), returned as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the named output dtype ('f32' or 'bf16'), returned as float64."""
    if dtype == "f32":
        return round_f32(x)
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")
