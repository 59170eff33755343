"""Storage formats and the rounding rho.  TEST INFRASTRUCTURE ONLY (see package doc).

bfloat16 keeps the float32 sign and 8-bit exponent and 7 stored mantissa bits.
Decoding a bf16 bit pattern is exact: the 16 bits are the upper half of a
float32.  Encoding rounds a real value to the nearest bf16, ties to even.
"""
from __future__ import annotations

import numpy as np


def bf16_decode(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_bf16(v: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    Returns float64 values that are exactly representable in bf16.  Written
    from the format definition: a normal bf16 value has 8 significant bits, so
    for |v| in [2^(e-1), 2^e) the spacing of representable values is 2^(e-8);
    below the smallest normal 2^-126 the spacing stays 2^-133 (subnormals).
    Values past the largest finite bf16 round to +-inf.
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros_like(v)
    nz = (v != 0) & np.isfinite(v)
    _, e = np.frexp(v[nz])                       # v = m * 2^e, 0.5 <= |m| < 1
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)   # spacing at that binade
    r = np.rint(v[nz] / q) * q                   # rint: round half to even
    bf16_max = (2.0 - 2.0 ** -7) * 2.0 ** 127
    r[np.abs(r) > bf16_max] = np.copysign(np.inf, r[np.abs(r) > bf16_max])
    out[nz] = r
    out[~np.isfinite(v)] = v[~np.isfinite(v)]
    out[v == 0] = v[v == 0]                      # keeps the sign of zero
    return out


def bf16_encode(v: np.ndarray) -> np.ndarray:
    """float64 -> uint16 bf16 bit patterns (round to nearest even)."""
    r = round_bf16(v).astype(np.float32)         # exact: r is a bf16 value
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def decode(a: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array -> float64 values ("f32": float32 array, "bf16": uint16 bits)."""
    if dtype == "bf16":
        return bf16_decode(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def rho(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the activation storage type; returns float64 values."""
    if dtype == "bf16":
        return round_bf16(v)
    if dtype == "f32":
        return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(dtype)
