"""Storage dtypes and round-to-nearest-even narrowing (oracle).

The paper does not state the KV precision (App. B.2 quantises weights only),
so the storage dtype is a parameter: ``"f32"`` (IEEE binary32) or ``"bf16"``
(bfloat16: binary32 with the low 16 bits dropped).  Every narrowing rounds to
nearest, ties to even, from the exact float64 value in ONE step (no double
rounding through fp32).

bf16 tensors travel as ``uint16`` bit patterns; fp32 tensors as ``float32``.

Pins (tests/test_oracle_numerics.py): agreement with torch's fp32->bf16
conversion on random and tie-heavy fp32 inputs; for float64 inputs, the result
is the nearer of the two bf16 neighbours (even mantissa on a tie), found by
enumeration.
"""
from __future__ import annotations

import numpy as np

DTYPES = ("f32", "bf16")

# bfloat16: 8 significant bits, exponent range of binary32.
_BF16_MANT_BITS = 8
_BF16_MIN_EXP = -133          # 2^-133 is the smallest subnormal step
_BF16_MAX = float(np.float32(3.3895313892515355e38))


def bf16_round(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    # quantum of the bf16 grid at this binade (subnormal floor applied)
    q = np.maximum(e - _BF16_MANT_BITS, _BF16_MIN_EXP)
    y = np.ldexp(np.rint(np.ldexp(x, -q)), q)   # rint: ties to even; scaling is exact
    y = np.where(np.abs(y) > _BF16_MAX, np.copysign(np.inf, x), y)
    return np.where(np.isfinite(x), y, x)


def bf16_bits(x_bf16_valued) -> np.ndarray:
    """uint16 bit pattern of values that are already bf16-representable."""
    f = np.asarray(x_bf16_valued, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_value(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def decode(arr, dtype: str) -> np.ndarray:
    """Storage array -> float64 values."""
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_value(arr)
    raise ValueError(dtype)


def round_to(x, dtype: str) -> np.ndarray:
    """float64 -> nearest storage value, returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)   # IEEE RNE, single rounding
    if dtype == "bf16":
        return bf16_round(x)
    raise ValueError(dtype)


def encode(x, dtype: str) -> np.ndarray:
    """float64 -> storage array (rounding first)."""
    r = round_to(x, dtype)
    if dtype == "f32":
        return r.astype(np.float32)
    return bf16_bits(r)


def ulp(x_storage_valued, dtype: str) -> np.ndarray:
    """Spacing of the storage grid at |x| (the gap to the next value away from 0)."""
    x = np.abs(np.asarray(x_storage_valued, dtype=np.float64))
    mant = 24 if dtype == "f32" else _BF16_MANT_BITS
    min_exp = -149 if dtype == "f32" else _BF16_MIN_EXP
    _, e = np.frexp(x)
    return np.ldexp(1.0, np.maximum(e - mant, min_exp))
