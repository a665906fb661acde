"""Rotary embedding of query/key vectors (Section 3.1 and Appendix A.5 of the paper).

For one token and one head, pair j = 0..D/2-1 is (x[2j], x[2j+1]) (interleaved
pairs).  With that token's cached coefficients c = cos, s = sin for pair j:

    y[2j]   = x[2j] * c - x[2j+1] * s
    y[2j+1] = x[2j] * s + x[2j+1] * c

which is the complex product (x[2j] + i x[2j+1]) * exp(i * angle).  The paper
states the arithmetic is the whole computation: bf16 inputs are widened to
fp32, rotated in fp32 with fp32 tables, and stored back as bf16.

Rounding contract (the paper fixes fp32 math but not the operation order or
contraction): every product and the sum/difference are separate IEEE binary32
operations rounded to nearest-even (no fused multiply-add), and the result is
rounded to bf16 nearest-even:

    y_e = bf16( f32( f32(x_e*c) - f32(x_o*s) ) )
    y_o = bf16( f32( f32(x_e*s) + f32(x_o*c) ) )

Emulated here in float64: a bf16 x binary32 product has at most 8 + 24
significant bits, so it is exact in float64 and rounding it to binary32 gives
the binary32 product; a float64 sum of two binary32 values rounded to binary32
equals the binary32 sum because 53 >= 2*24 + 2 makes the double rounding
harmless.  ``tests/test_oracle_rope.py`` also checks this against NumPy's own
float32 arithmetic.
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_to_f64, f32_to_bf16_bits, f32_to_f64, round_f32


def _broadcast_tables(t: np.ndarray, x_shape) -> np.ndarray:
    """Table [N, P] -> shape broadcastable to x[..., N, H, P] (shared across heads)."""
    t = np.asarray(t)
    n, p = t.shape
    lead = len(x_shape) - 3
    return t.reshape((1,) * lead + (n, 1, p))


def rope_bf16(x_bits: np.ndarray, cos32: np.ndarray, sin32: np.ndarray) -> np.ndarray:
    """Rotate bf16 vectors x[..., N, H, D] with fp32 tables [N, D/2]; returns bf16 bits.

    Follows the rounding contract in the module docstring.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    xe = bf16_to_f64(x_bits[..., 0::2])
    xo = bf16_to_f64(x_bits[..., 1::2])
    c = _broadcast_tables(f32_to_f64(cos32), x_bits.shape)
    s = _broadcast_tables(f32_to_f64(sin32), x_bits.shape)
    ye = round_f32(round_f32(xe * c) - round_f32(xo * s))
    yo = round_f32(round_f32(xe * s) + round_f32(xo * c))
    y = np.empty(x_bits.shape, dtype=np.uint16)
    y[..., 0::2] = f32_to_bf16_bits(ye)
    y[..., 1::2] = f32_to_bf16_bits(yo)
    return y


def rope_ideal(x: np.ndarray, angles: np.ndarray) -> np.ndarray:
    """Exact-arithmetic rotation in float64 (no intermediate rounding, float64 angles).

    x[..., N, H, D] float64, angles [N, D/2] float64.  Used for the invariants
    (norm preservation, relative-position property).
    """
    x = np.asarray(x, dtype=np.float64)
    a = _broadcast_tables(angles, x.shape)
    c, s = np.cos(a), np.sin(a)
    xe, xo = x[..., 0::2], x[..., 1::2]
    y = np.empty_like(x)
    y[..., 0::2] = xe * c - xo * s
    y[..., 1::2] = xe * s + xo * c
    return y
