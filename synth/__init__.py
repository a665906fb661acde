"""Seeded synthetic inputs for the windowed-attention chunk step.

This module is shared by the tests, the bench and the oracle's checks, so it
deliberately holds none of the step's arithmetic: no rotary embedding, no slot
mapping, no attention.  It only

* names the workloads (shapes of the causal video DiT's self-attention step:
  12 heads of width 128, 30x52 = 1560 tokens per latent frame, 3-frame chunks;
  the paper's Appendix A.1 and A.5 fix these), and
* draws seeded N(0,1) values and rounds them to bfloat16 bit patterns.

Every random draw comes from NumPy's PCG64 seeded by a SeedSequence whose key
starts with (2609, 32518) and continues with the caller's key, so a tensor is
identified by e.g. (config, layer, chunk, pass, tensor-id).
"""
from __future__ import annotations

import dataclasses
from typing import Tuple

import numpy as np

# tensor ids inside a seed key
Q, K, V, CACHE_K, CACHE_V = 0, 1, 2, 3, 4


def generator(*key: int) -> np.random.Generator:
    """PCG64 generator for the seed key (2609, 32518, *key)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([2609, 32518, *[int(k) for k in key]])))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 draws to the nearest bfloat16 (ties to even); returns uint16 bits.

    Used only to turn random draws into bf16 inputs; NaN never occurs here.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    # finite values stay below 2^32 - 0x8000 after the increment, so 32 bits suffice
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return u.astype(np.uint16)


def normal_bf16(shape: Tuple[int, ...], key: Tuple[int, ...], scale: float = 1.0) -> np.ndarray:
    """Seeded N(0, scale^2) draw, rounded to bf16, as uint16 bits of the given shape."""
    g = generator(*key)
    x = g.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x = (x * np.float32(scale)).astype(np.float32)
    return bf16_bits_from_f32(x)


def normal_f32(shape: Tuple[int, ...], key: Tuple[int, ...], scale: float = 1.0) -> np.ndarray:
    """Seeded N(0, scale^2) float32 draw (e.g. a projection weight before its bf16 cast)."""
    x = generator(*key).standard_normal(size=shape, dtype=np.float32)
    return (x * np.float32(scale)).astype(np.float32) if scale != 1.0 else x


def small_int_bf16(shape: Tuple[int, ...], values: np.ndarray) -> np.ndarray:
    """bf16 bits of small exact integers (|v| < 256), broadcast to `shape`."""
    v = np.broadcast_to(np.asarray(values, dtype=np.float32), shape)
    return bf16_bits_from_f32(v)


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shapes of one chunk-step workload.

    B batch, H heads, D head width, (grid_h, grid_w) latent token grid (T =
    grid_h*grid_w tokens per frame), C frames per chunk, S sink frames, W prior
    window frames, R ring frames, f0 the chunk's start frame (for streams: the
    first chunk), theta the rotary base.
    """
    name: str
    B: int
    H: int
    D: int
    grid_h: int
    grid_w: int
    C: int
    S: int
    W: int
    R: int
    f0: int
    theta: float = 10000.0
    layers: int = 1          # distinct per-layer caches (short window + refine)
    passes: int = 1          # calls per chunk per layer (denoise + clean-cache refine)
    chunks: int = 1          # consecutive chunks (rolling stream)

    @property
    def T(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def n_query(self) -> int:
        return self.C * self.T

    @property
    def slots(self) -> int:
        return (self.S + self.R) * self.T

    def prior_starts(self):
        """Start frames of the C-frame chunks appended before the measured chunk
        (frames 0 .. f0-1, in chunk order) to fill the cache through the library."""
        return list(range(0, self.f0, self.C))


WORKLOADS = {
    # 2 heads, 4x6 grid, 3-frame chunk at frame 6 over 6 prior frames
    "tiny": Workload("tiny", B=1, H=2, D=128, grid_h=4, grid_w=6, C=3, S=0, W=6, R=9, f0=6),
    # 12x128 heads, 30x52 grid, 3-frame chunk (4680 queries) at frame 9 over 9 prior frames
    "full_chunk": Workload("full_chunk", B=1, H=12, D=128, grid_h=30, grid_w=52, C=3, S=0, W=9, R=12, f0=9),
    # same shapes, every one of 18 prior frames kept (32760 keys)
    "unwindowed": Workload("unwindowed", B=1, H=12, D=128, grid_h=30, grid_w=52, C=3, S=0, W=18, R=21, f0=18),
    # 3 prior frames (9360 keys), two calls per chunk, 30 layers with their own caches
    "short_refine": Workload("short_refine", B=1, H=12, D=128, grid_h=30, grid_w=52, C=3, S=0, W=3, R=6, f0=12,
                             layers=30, passes=2),
    # 1-frame chunks, 60 of them through a 12-frame ring
    "rolling": Workload("rolling", B=1, H=12, D=128, grid_h=30, grid_w=52, C=1, S=0, W=11, R=12, f0=0, chunks=60),
    # the paper's own default window: 3 sink frames + 6 recent frames including the chunk (14040 keys)
    "paper_default": Workload("paper_default", B=1, H=12, D=128, grid_h=30, grid_w=52, C=3, S=3, W=3, R=6, f0=9),
}
