"""Rounding helpers for the oracle.

Every operator is evaluated in float64 and its result rounded to the edge's
storage type: float32 by round-to-nearest-even (numpy's cast), bfloat16 as
float64 -> float32 -> bfloat16, both steps round-to-nearest-even.  bfloat16
is the top 16 bits of a float32; rounding is done on the bit pattern since
numpy has no bfloat16 type.  Values are carried as float64 arrays that hold
exactly representable float32 / bfloat16 numbers.
"""
from __future__ import annotations

import numpy as np


def f32_to_bf16_bits(a) -> np.ndarray:
    """float32 array -> uint16 bfloat16 bit patterns, round-to-nearest-even.

    NaN maps to the quiet NaN 0x7FC0 (sign kept); +-inf stays +-inf; finite
    values past the largest bfloat16 round to +-inf as RNE requires.
    """
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        sign = ((u >> np.uint64(16)) & np.uint64(0x8000)).astype(np.uint16)
        r = np.where(nan, sign | np.uint16(0x7FC0), r)
    return r


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_f32(a) -> np.ndarray:
    """float64 -> nearest float32 (RNE), returned as float64."""
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_bf16(a) -> np.ndarray:
    """float64 -> float32 (RNE) -> bfloat16 (RNE), returned as float64."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    return bf16_bits_to_f32(f32_to_bf16_bits(f)).astype(np.float64)


def round_to(a, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return round_f32(a)
    if dtype == "bf16":
        return round_bf16(a)
    raise ValueError(dtype)


def itemsize(dtype: str) -> int:
    return {"f32": 4, "bf16": 2}[dtype]


def to_bytes(a, dtype: str) -> np.ndarray:
    """float64 array of representable values -> raw little-endian bytes (uint8)."""
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32).view(np.uint8).ravel()
    return f32_to_bf16_bits(np.asarray(a, np.float32)).view(np.uint8).ravel()


def from_bytes(buf, dtype: str, count: int) -> np.ndarray:
    """raw bytes -> float64 array of ``count`` elements."""
    buf = np.ascontiguousarray(buf, dtype=np.uint8)
    if dtype == "f32":
        return buf[: 4 * count].view(np.float32).astype(np.float64)
    return bf16_bits_to_f32(buf[: 2 * count].view(np.uint16)).astype(np.float64)
