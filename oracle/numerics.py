"""Bit-level number formats used by the oracle (bfloat16 and IEEE binary32).

bf16 values are carried as uint16 bit patterns; conversions are written out
from the format definitions (bf16 = the upper 16 bits of a binary32).
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns as float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def f32_to_f64(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def round_f32(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest binary32 (ties to even), kept as float64.

    NumPy's float64 -> float32 cast is the IEEE round-to-nearest-even conversion.
    """
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary32 values (given exactly as float64 or float32) to bf16, ties to even.

    Integer form of round-to-nearest-even on the binary32 bit pattern: add
    0x7FFF plus the lowest kept bit, then drop the low 16 bits.  NaN inputs are
    not supported (the step never produces them from finite inputs).
    """
    f = np.asarray(x).astype(np.float32)
    if not np.all(np.isfinite(f)):
        raise ValueError("non-finite value reached bf16 rounding")
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    return ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
