"""Sink + sliding-window KV cache with host-held indices (paper Sections 3.1, 3.3;
Appendix A.3 and A.5).

The paper keeps the first latent frames as attention sinks and a window of the
most recent frames, evicting the middle; the cache positions are host integers
that depend only on token positions and counts, and a repeated denoising call
for the same chunk overwrites that chunk's entries without advancing them.

Model used here (readings where the paper is silent):

* eviction is by whole latent frames; S sink slots hold frames 0..S-1, and R
  ring slots hold the other frames: frame f < S lives in slot f, frame f >= S
  in slot S + (f - S) mod R; token t of a frame lives at row slot*T + t;
* the keys retained for a chunk of C frames starting at f0 with a window of W
  prior frames are the sinks older than the window, then the W frames before
  f0, then the chunk itself: frames [0, min(S, lo)) + [lo, f0 + C) with
  lo = max(0, f0 - W), in that (logical) order;
* block-causal masking with the chunk as the block: every query of the chunk
  sees every retained key (the chunk's own keys included), nothing later.

The cache is simulated with a plain per-slot store; errors use four kinds that
mirror the library's status codes: "shape", "range", "state" (and "null",
which cannot arise in Python).
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np


class OracleError(Exception):
    def __init__(self, kind: str, msg: str):
        super().__init__(f"{kind}: {msg}")
        self.kind = kind


def slot_of_frame(f: int, S: int, R: int) -> int:
    return f if f < S else S + (f - S) % R


def retained_frames(f0: int, C: int, S: int, W: int) -> List[int]:
    lo = max(0, f0 - W)
    return list(range(0, min(S, lo))) + list(range(lo, f0 + C))


class KVCacheOracle:
    """K/V cache of one attention layer: bf16 bits [B, H, (S+R)*T, D] plus host indices."""

    def __init__(self, B: int, H: int, D: int, grid_h: int, grid_w: int, S: int, R: int):
        if min(B, H, D, grid_h, grid_w) < 1 or S < 0 or R < 1:
            raise OracleError("shape", "bad cache geometry")
        self.B, self.H, self.D = B, H, D
        self.T = grid_h * grid_w
        self.S, self.R = S, R
        self.k = np.zeros((B, H, (S + R) * self.T, D), dtype=np.uint16)
        self.v = np.zeros_like(self.k)
        self.frame_of_slot = [-1] * (S + R)
        self.newest = -1

    # -- indices ---------------------------------------------------------
    def slot(self, f: int) -> int:
        return slot_of_frame(f, self.S, self.R)

    def resident(self, f: int) -> bool:
        return f >= 0 and self.frame_of_slot[self.slot(f)] == f

    def _check_append(self, f0: int, C: int) -> None:
        if C < 1:
            raise OracleError("shape", "empty chunk")
        if f0 < 0:
            raise OracleError("range", "negative start frame")
        ring_frames = sum(1 for f in range(f0, f0 + C) if f >= self.S)
        if ring_frames > self.R:
            raise OracleError("range", "chunk larger than the ring")
        if f0 > self.newest + 1:
            raise OracleError("state", "gap before the chunk")
        for f in range(f0, f0 + C):
            if f <= self.newest and not self.resident(f):
                raise OracleError("state", f"frame {f} was evicted")

    def append(self, f0: int, C: int, k_rot: np.ndarray, v: np.ndarray) -> None:
        """Write the chunk's rotated keys and values (bf16 bits [B, C*T, H, D])."""
        self._check_append(f0, C)
        T = self.T
        assert k_rot.shape == (self.B, C * T, self.H, self.D) and v.shape == k_rot.shape
        for i in range(C):
            f = f0 + i
            s = self.slot(f)
            rows = slice(s * T, (s + 1) * T)
            self.k[:, :, rows, :] = np.transpose(k_rot[:, i * T:(i + 1) * T], (0, 2, 1, 3))
            self.v[:, :, rows, :] = np.transpose(v[:, i * T:(i + 1) * T], (0, 2, 1, 3))
            self.frame_of_slot[s] = f
        self.newest = max(self.newest, f0 + C - 1)

    def retained(self, f0: int, C: int, W: int) -> List[int]:
        if C < 1:
            raise OracleError("shape", "empty chunk")
        if f0 < 0 or W < 0:
            raise OracleError("range", "negative start frame or window")
        frames = retained_frames(f0, C, self.S, W)
        if sum(1 for f in frames if f >= self.S) > self.R:
            raise OracleError("range", "window plus chunk larger than the ring")
        for f in frames:
            if not self.resident(f):
                raise OracleError("state", f"frame {f} is not in the cache")
        return frames

    def key_rows(self, f0: int, C: int, W: int) -> np.ndarray:
        """Physical cache rows of the retained keys, in logical order."""
        T = self.T
        frames = self.retained(f0, C, W)
        return np.concatenate([self.slot(f) * T + np.arange(T) for f in frames]).astype(np.int64)

    def segments(self, f0: int, C: int, W: int) -> List[Tuple[int, int]]:
        """Retained rows as maximal runs of consecutive physical rows: [(row0, length)]."""
        rows = self.key_rows(f0, C, W)
        segs: List[Tuple[int, int]] = []
        start = prev = int(rows[0])
        for r in rows[1:]:
            r = int(r)
            if r != prev + 1:
                segs.append((start, prev - start + 1))
                start = r
            prev = r
        segs.append((start, prev - start + 1))
        return segs
