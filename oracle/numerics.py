"""Exact rounding helpers for the oracle (test infrastructure only).

Representation: float32 tensors are numpy float32 arrays; bfloat16 tensors
are numpy uint16 arrays holding the bit pattern (sign, 8-bit exponent, 7-bit
fraction -- the upper half of an IEEE binary32).

Rounding is round-to-nearest, ties-to-even, applied once from the float64
value to the output format, with the binary32 exponent range (bfloat16
shares it): overflow goes to infinity, tiny values to subnormals.
"""
from __future__ import annotations

import numpy as np

F32 = "f32"
BF16 = "bf16"

_BF16_QEXP_MIN = -133     # quantum of bf16 subnormals: 2^-126 * 2^-7


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> exact float64 values."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x) -> np.ndarray:
    """float64 -> bf16 bits, one round-to-nearest-even step.

    The value is split as a = q * 2^e with e the exponent of its unit in the
    last place (7 fraction bits below the leading bit, never below the
    subnormal quantum 2^-133); q is rounded to an integer with ties to even
    (numpy.rint) and scaled back, which is exact in float64.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    with np.errstate(over="ignore", invalid="ignore"):
        finite = np.isfinite(a)
        af = np.where(finite, a, 0.0)
        _, e = np.frexp(af)                      # af = m * 2^e, m in [0.5, 1)
        qexp = np.maximum(e - 8, _BF16_QEXP_MIN)
        q = np.ldexp(af, -qexp)
        r = np.rint(q)                           # ties to even
        val = np.ldexp(r, qexp)
        f = val.astype(np.float32)               # exact, or +inf past the range
    mag = (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    mag = np.where(np.isinf(a), np.uint16(0x7F80), mag)
    mag = np.where(np.isnan(a), np.uint16(0x7FC0), mag)
    sign = np.where(np.signbit(x), np.uint16(0x8000), np.uint16(0))
    return (mag | sign).astype(np.uint16)


def f64_to_f32(x) -> np.ndarray:
    """float64 -> float32 with round-to-nearest-even (numpy's cast)."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float32)


def values(a: np.ndarray, dtype: str) -> np.ndarray:
    """Tensor in its storage representation -> exact float64 values."""
    if dtype == BF16:
        return bf16_bits_to_f64(a)
    if dtype == F32:
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage representation of `dtype`, rounded once."""
    if dtype == BF16:
        return f64_to_bf16_bits(x)
    if dtype == F32:
        return f64_to_f32(x)
    raise ValueError(dtype)


def bf16_ulp_distance(a_bits: np.ndarray, b_bits: np.ndarray) -> np.ndarray:
    """Number of representable bf16 values between two bit patterns.

    Maps the sign-magnitude patterns onto a monotone integer line, so +0 and
    -0 are distance 0 apart and adjacent values distance 1.
    """
    def line(bits):
        b = np.asarray(bits, dtype=np.uint16).astype(np.int64)
        mag = b & 0x7FFF
        return np.where(b & 0x8000, -mag, mag)
    return np.abs(line(a_bits) - line(b_bits))
