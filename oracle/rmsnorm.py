"""RMS normalisation of a token's query or key vector before RoPE (Appendix A.5 of the paper).

The paper's model reshapes each query and newly computed key into heads *after* the
linear projection and an RMS normalisation, so the normalisation runs over all H*D
channels of one token (1536 for 12 heads of width 128), with a learned per-channel
weight w:

    y_j = x_j * w_j / sqrt( (1/C) * sum_i x_i^2 + eps ),   C = H * D

The paper does not give eps or the precision.  Readings taken here: eps = 1e-6; the
statistic and the scale in float64; the result rounded once to binary32 and then to
bf16 (nearest-even both times), since the rotary kernel that follows takes bf16:

    ss  = sum_i x_i^2                           (float64)
    r   = 1 / sqrt(ss / C + eps)                (float64, correctly rounded sqrt and division)
    y_j = bf16( f32( (x_j * r) * w_j ) )        (float64 products)

Every square of a bf16 value is exact in float64, so ss is exact (here summed with
math.fsum, i.e. exactly rounded) whenever the squares span less than about 2^26; the
GPU's float64 sum in another order can then differ only in its last bit, which changes
the bf16 result only if the product lands within ~2^-52 of a rounding midpoint.

Test infrastructure: nothing in the library imports this module.
"""
from __future__ import annotations

import math

import numpy as np

from .numerics import bf16_to_f64, f32_to_bf16_bits, round_f32

EPS = 1e-6


def rms_norm_bf16(x_bits: np.ndarray, w_bits: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Normalise bf16 vectors x[..., C] (last axis = the token's channels) with bf16 weights
    w[C]; returns bf16 bits of the same shape, following the contract in the module docstring.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    w = bf16_to_f64(np.asarray(w_bits, dtype=np.uint16))
    if w.shape != x_bits.shape[-1:]:
        raise ValueError(f"weight shape {w.shape} does not match channels {x_bits.shape[-1:]}")
    x = bf16_to_f64(x_bits)
    C = x.shape[-1]
    flat = x.reshape(-1, C)
    ss = np.array([math.fsum(row * row) for row in flat]).reshape(x.shape[:-1] + (1,))
    r = 1.0 / np.sqrt(ss / C + eps)
    return f32_to_bf16_bits(round_f32((x * r) * w))


def rms_norm_ideal(x: np.ndarray, w: np.ndarray, eps: float = EPS) -> np.ndarray:
    """The same normalisation in float64 throughout, no rounding of the result."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(w, dtype=np.float64)


def split_heads(x_bits: np.ndarray, heads: int) -> np.ndarray:
    """Token vectors [..., N, H*D] -> [..., N, H, D] (the reshape into heads)."""
    x_bits = np.asarray(x_bits)
    return x_bits.reshape(x_bits.shape[:-1] + (heads, x_bits.shape[-1] // heads))
