"""Per-chunk 3D rotary cos/sin tables (Appendix A.5 of the paper).

The paper builds, once per (start latent frame, grid size), fp32 cos and sin
tables holding one coefficient per token and coordinate pair, shared by all
heads; each token's coefficients combine its frame, row and column positions.
The chunk starting at latent frame 6 uses temporal positions 6, 7, 8.

Readings taken where the paper is silent:

* split of the D/2 pairs over the three axes: the height and width axes take
  2*(D//6) dimensions each and the temporal axis the rest, in the order
  (temporal, height, width); for D = 128 that is 22 / 21 / 21 pairs
  (44 / 42 / 42 dimensions);
* frequency ladder per axis: omega_k = 1 / theta**((2k)/d_axis) for
  k = 0 .. d_axis/2 - 1, evaluated in float64 with the C library's pow;
* positions: absolute latent frame index for time, 0-based token-grid row and
  column for space;
* token order inside a chunk: frame-major, then row, then column;
* angle = position * omega in float64; cos and sin in float64 with the C
  library, then rounded once to binary32.

Python's ``math`` module calls the platform C library, so these values are
what a C++ host computing the same expressions with ``std::pow/cos/sin``
obtains on the same machine.
"""
from __future__ import annotations

import math
from typing import List, Tuple

import numpy as np

TEMPORAL, HEIGHT, WIDTH = 0, 1, 2


def axis_dims(head_dim: int) -> Tuple[int, int, int]:
    """(d_t, d_h, d_w): dimensions of the head vector given to each axis."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    d_h = d_w = 2 * (head_dim // 6)
    d_t = head_dim - d_h - d_w
    return d_t, d_h, d_w


def pair_axes(head_dim: int) -> List[Tuple[int, int, int]]:
    """For each pair j = 0 .. head_dim/2 - 1: (axis, k, d_axis)."""
    d_t, d_h, d_w = axis_dims(head_dim)
    out = []
    for axis, d_ax in ((TEMPORAL, d_t), (HEIGHT, d_h), (WIDTH, d_w)):
        for k in range(d_ax // 2):
            out.append((axis, k, d_ax))
    assert len(out) == head_dim // 2
    return out


def omega(theta: float, k: int, d_axis: int) -> float:
    """Rotation frequency of ladder step k on an axis of d_axis dimensions."""
    return 1.0 / math.pow(theta, (2.0 * k) / d_axis)


def token_positions(start_frame: int, n_frames: int, grid_h: int, grid_w: int) -> np.ndarray:
    """[N, 3] int64 (frame, row, column) of each chunk token, frame-major order."""
    f, h, w = np.meshgrid(np.arange(n_frames), np.arange(grid_h), np.arange(grid_w), indexing="ij")
    pos = np.stack([f.ravel() + start_frame, h.ravel(), w.ravel()], axis=1)
    return pos.astype(np.int64)


def angles_f64(start_frame: int, n_frames: int, grid_h: int, grid_w: int, head_dim: int,
               theta: float) -> np.ndarray:
    """[N, head_dim/2] float64 angle p_axis * omega_k of every token and pair."""
    pos = token_positions(start_frame, n_frames, grid_h, grid_w)
    axes = pair_axes(head_dim)
    ang = np.empty((pos.shape[0], len(axes)), dtype=np.float64)
    for j, (axis, k, d_ax) in enumerate(axes):
        w = omega(theta, k, d_ax)
        for n in range(pos.shape[0]):
            ang[n, j] = float(pos[n, axis]) * w
    return ang


def rope_tables(start_frame: int, n_frames: int, grid_h: int, grid_w: int, head_dim: int = 128,
                theta: float = 10000.0) -> Tuple[np.ndarray, np.ndarray]:
    """cos, sin tables: float32 arrays of shape [n_frames*grid_h*grid_w, head_dim/2].

    Each entry is binary32(cos(angle)) / binary32(sin(angle)) with the angle and
    the trigonometric function evaluated in float64.  Distinct angles are few
    (one per axis position and ladder step), so each is evaluated once and the
    token rows are gathered from those values.
    """
    pos = token_positions(start_frame, n_frames, grid_h, grid_w)
    axes = pair_axes(head_dim)
    cos_t = np.empty((pos.shape[0], len(axes)), dtype=np.float32)
    sin_t = np.empty_like(cos_t)
    for j, (axis, k, d_ax) in enumerate(axes):
        w = omega(theta, k, d_ax)
        col = pos[:, axis]
        memo_c, memo_s = {}, {}
        for p in np.unique(col):
            a = float(p) * w
            memo_c[int(p)] = np.float32(math.cos(a))
            memo_s[int(p)] = np.float32(math.sin(a))
        cos_t[:, j] = [memo_c[int(p)] for p in col]
        sin_t[:, j] = [memo_s[int(p)] for p in col]
    return cos_t, sin_t
