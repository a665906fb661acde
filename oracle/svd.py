"""Truncated SVD of the attention value and output projections, and the projection after
attention (Section 3.5, Equation for the rank-r reconstruction, and Appendix A.4).

For W in R^{m x n} with W = U S V^T (singular values in decreasing order), the edit keeps the
r leading directions, W_r = U_r S_r V_r^T, stored densely in W's shape.  The model's 1536 x
1536 value and output weights of layers 8-29 (of 30) are replaced at r = round(0.92 * 1536) =
1413; queries, keys and layers 0-7 keep their weights.  The paper computes the decomposition
and the reconstruction in float32 and then casts the model to bf16.

Here W_r is the exact definition evaluated in float64 (LAPACK's SVD of the float32 matrix,
which float64 holds exactly, as the decomposition step); the stored weight is that value
rounded to float32 and then to bf16, both nearest-even (the paper's float32 reconstruction
cast to bf16).  The projection y = x W^T + b (nn.Linear layout: W is [out, in]) is exact
in float64 on the bf16 operands.

Test infrastructure: nothing in the library imports this module.
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_to_f64, f32_to_bf16_bits

RETAIN = 0.92
FIRST_TRUNCATED_LAYER = 8
N_LAYERS = 30


def rank_for(m: int, retain: float = RETAIN) -> int:
    """r = round(retain * m), m = the smaller dimension."""
    return int(np.floor(retain * m + 0.5))


def truncated_layers(n_layers: int = N_LAYERS, first: int = FIRST_TRUNCATED_LAYER):
    return list(range(first, n_layers))


def singular_values(w: np.ndarray) -> np.ndarray:
    return np.linalg.svd(np.asarray(w, dtype=np.float64), compute_uv=False)


def truncate(w: np.ndarray, rank: int) -> np.ndarray:
    """W_r = U_r S_r V_r^T in float64."""
    w = np.asarray(w, dtype=np.float64)
    if not 0 <= rank <= min(w.shape):
        raise ValueError("rank must lie in [0, min(m, n)]")
    u, s, vt = np.linalg.svd(w, full_matrices=False)
    return (u[:, :rank] * s[:rank]) @ vt[:rank]


def truncate_bf16(w: np.ndarray, rank: int) -> np.ndarray:
    """The stored weight: W_r rounded to bf16 (bits)."""
    return f32_to_bf16_bits(truncate(w, rank))


def linear(x_bits: np.ndarray, w_bits: np.ndarray, b_bits=None) -> np.ndarray:
    """y = x W^T + b in float64 for bf16 x [..., K], W [N, K], b [N]."""
    x = bf16_to_f64(np.asarray(x_bits, dtype=np.uint16))
    w = bf16_to_f64(np.asarray(w_bits, dtype=np.uint16))
    if w.ndim != 2 or x.shape[-1] != w.shape[1]:
        raise ValueError("x [..., K] and W [N, K] required")
    y = x @ w.T
    if b_bits is not None:
        y = y + bf16_to_f64(np.asarray(b_bits, dtype=np.uint16))
    return y
