"""bfloat16 rounding for the oracle, written from the IEEE-754 definition.

bf16 keeps float32's 8-bit exponent and 7 stored fraction bits (8 significant
bits). A finite value x is rounded to the nearest representable bf16 value,
ties going to the one whose last significand bit is 0 (round to nearest even),
the rounding the paper applies when it stores bf16 activations (Appendix A,
TwELL matmul). This module does that with fp64 arithmetic on the exact value:
scale by the bf16 unit in the last place of x's binade, round half to even,
scale back. Subnormals are kept (no flush), overflow goes to infinity, NaN
stays NaN.
"""
from __future__ import annotations

import numpy as np

_EMIN = -126        # smallest normal exponent
_P = 8              # significant bits of bf16
_MAX_FINITE = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_to_bf16_value(x) -> np.ndarray:
    """Return the bf16 value nearest to x (float64 array holding exact bf16 values)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, dtype=np.float64, copy=True)
    finite = np.isfinite(x) & (x != 0)
    xf = x[finite]
    mant, exp = np.frexp(np.abs(xf))      # |x| = mant * 2**exp, mant in [0.5, 1)
    e = np.maximum(exp - 1, _EMIN)        # binade exponent, clamped to the subnormal range
    ulp = np.ldexp(1.0, e - (_P - 1))
    r = np.rint(xf / ulp) * ulp           # np.rint rounds half to even
    r = np.where(np.abs(r) > _MAX_FINITE, np.inf, r)
    out[finite] = np.copysign(r, xf)
    return out


def bits_of_bf16_value(v) -> np.ndarray:
    """Bit pattern (uint16) of values that are already exact bf16 values."""
    v = np.asarray(v, dtype=np.float64)
    f32 = v.astype(np.float32)            # exact: every bf16 value is a float32 value
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    return np.where(np.isnan(v), np.uint16(0x7FC0), bits)


def to_bf16_bits(x) -> np.ndarray:
    return bits_of_bf16_value(round_to_bf16_value(x))


def from_bf16_bits(b) -> np.ndarray:
    """Exact float64 value of bf16 bit patterns."""
    b = np.asarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
