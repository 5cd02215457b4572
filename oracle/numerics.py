"""Storage-type conversions used by the oracle.

bf16 is carried as uint16 bit patterns.  Rounding fp32 -> bf16 is
round-to-nearest, ties-to-even on the 16 dropped bits (IEEE 754 default
rounding applied to the bfloat16 format: 1 sign, 8 exponent, 7 fraction bits).
NaN stays NaN (quiet bit forced).

Pinned in tests/test_oracle_numerics.py against hand-computed bit patterns
(ties, carries into the exponent, overflow to infinity) and against torch's
own float32 -> bfloat16 conversion on random data.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    u16 = np.asarray(u16, dtype=np.uint16)
    return (u16.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(f: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(f, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    r = np.where(nan, (u >> np.uint64(16)) | np.uint64(0x40), r)
    return (r & np.uint64(0xFFFF)).astype(np.uint16)


def storage_to_f32(a: np.ndarray) -> np.ndarray:
    """Storage array (float32, or uint16 bf16 bits) -> float32 (exact)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_bits_to_f32(a)
    if a.dtype == np.float32:
        return a
    raise TypeError(f"unsupported storage dtype {a.dtype}")


def storage_to_f64(a: np.ndarray) -> np.ndarray:
    """Storage array -> float64 (exact)."""
    return storage_to_f32(a).astype(np.float64)


def f32_to_storage(f: np.ndarray, like: np.ndarray) -> np.ndarray:
    """Round float32 values to the storage type of ``like`` (identity for fp32)."""
    if np.asarray(like).dtype == np.uint16:
        return f32_to_bf16_bits(f)
    return np.ascontiguousarray(f, dtype=np.float32)


def f64_to_storage(f: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage: rounded to fp32 (RNE), then for bf16 to bf16 (RNE)."""
    f32 = np.asarray(f, dtype=np.float64).astype(np.float32)
    return f32_to_bf16_bits(f32) if dtype == "bf16" else f32
