"""Shared pieces of the GPU parity tests: bf16 bit transfer, a stream of chunk steps
driven through the library and mirrored by the oracle, and the attention tolerance.

Inputs come from ``synth`` only; expected values come from ``oracle`` only.
"""
from __future__ import annotations

import math
import sys
from typing import Optional, Sequence

import numpy as np
import torch

import synth
from oracle import attention, numerics, rmsnorm, rope, tables
from oracle.kvcache import KVCacheOracle

# attention tolerance stated for bf16 inputs with fp32 accumulation
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
# tighter relative bound: bf16 rounding of the output (<= 2^-9 relative) and of the
# probabilities fed to the PV product keep the mean error well under 2^-7 of the mean |o|
MEAN_REL = 2.0 ** -7
# log-sum-exp bound: the row sum adds fp32 probabilities, each within a few fp32 ulps of
# exp2 of the fp32 score (the hardware exp2 and the fp32 scores add a relative error far
# below 2^-9), so log(sum) moves by well under 2^-9; 2^-8 also covers a row sum built from
# the bf16-rounded probabilities (each within 2^-9 relative) should the kernel use them
LSE_ABS = 2.0 ** -8


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 bit patterns -> device bf16 tensor (same bits)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def host(t: torch.Tensor) -> np.ndarray:
    """device bf16 tensor -> uint16 bit patterns."""
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def check_attention(got_bits: np.ndarray, want: np.ndarray, what: str) -> dict:
    g = numerics.bf16_to_f64(got_bits)
    err = np.abs(g - want)
    stats = dict(max_abs=float(err.max()), mean_abs=float(err.mean()),
                 mean_rel=float(err.mean() / max(np.abs(want).mean(), 1e-30)),
                 rms_ref=float(np.sqrt(np.mean(want ** 2))))
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    assert stats["max_abs"] <= MAX_ABS, f"{what}: {stats}"
    assert stats["mean_abs"] <= MEAN_ABS, f"{what}: {stats}"
    assert stats["mean_rel"] <= MEAN_REL, f"{what}: {stats}"
    return stats


class Mirror:
    """A library cache and the oracle's cache driven by the same calls and inputs."""

    def __init__(self, u, B, H, grid_h, grid_w, S, R, device="cuda", guard_rows: int = 0):
        self.u = u
        self.B, self.H, self.gh, self.gw, self.S, self.R = B, H, grid_h, grid_w, S, R
        self.T = grid_h * grid_w
        self.slots = (S + R) * self.T
        self.guard = guard_rows
        if guard_rows:
            # cache rows live inside a larger buffer; the rows around them must stay untouched
            shape = (B * H * self.slots + 2 * guard_rows, 128)
            self.k_full = torch.full(shape, 1.5, dtype=torch.bfloat16, device=device)
            self.v_full = torch.full(shape, -2.5, dtype=torch.bfloat16, device=device)
            kc = self.k_full[guard_rows:guard_rows + B * H * self.slots].view(B, H, self.slots, 128)
            vc = self.v_full[guard_rows:guard_rows + B * H * self.slots].view(B, H, self.slots, 128)
            kc.zero_()
            vc.zero_()
            self.lib = u.Cache(B, H, grid_h, grid_w, S, R, device=device, k_cache=kc, v_cache=vc)
        else:
            self.lib = u.Cache(B, H, grid_h, grid_w, S, R, device=device)
        self.orc = KVCacheOracle(B, H, 128, grid_h, grid_w, S, R)
        self.tables = u.RopeTableCache(device)

    def inputs(self, C: int, key, q_scale=1.0, v_bits: Optional[np.ndarray] = None, q_zero=False,
               k_bits: Optional[np.ndarray] = None):
        shape = (self.B, C * self.T, self.H, 128)
        q = np.zeros(shape, np.uint16) if q_zero else synth.normal_bf16(shape, tuple(key) + (synth.Q,), q_scale)
        k = synth.normal_bf16(shape, tuple(key) + (synth.K,)) if k_bits is None else k_bits
        v = synth.normal_bf16(shape, tuple(key) + (synth.V,)) if v_bits is None else v_bits
        return q, k, v

    def skip_frames(self, f0: int, C: int) -> None:
        """Record frames as stored without data on both sides (their contents are evicted
        before they are ever read)."""
        self.lib.advance(f0, C)
        z = np.zeros((self.B, C * self.T, self.H, 128), np.uint16)
        self.orc.append(f0, C, z, z)

    def append(self, f0: int, C: int, key, with_q=False, **kw):
        q, k, v = self.inputs(C, key, **kw)
        cos_t, sin_t = self.tables.get(f0, C, self.gh, self.gw)
        qr = self.lib.unstep_kv_append(f0, C, dev(q) if with_q else None, dev(k), dev(v), cos_t, sin_t)
        c, s = tables.rope_tables(f0, C, self.gh, self.gw)
        self.orc.append(f0, C, rope.rope_bf16(k, c, s), v)
        return (q, qr, c, s) if with_q else None

    def append_qknorm(self, f0: int, C: int, key, wq_bits, wk_bits, eps=1e-6, with_q=True, q_layout="contiguous",
                      **kw):
        """unstep_kv_append_qknorm on both sides; returns (q_rot_dev, q_rot_oracle) (None, None without q)."""
        q, k, v = self.inputs(C, key, **kw)
        cos_t, sin_t = self.tables.get(f0, C, self.gh, self.gw)
        if q_layout == "fused_qkv":
            qkv = torch.stack([dev(q), dev(k), dev(v)], dim=2)       # [B, N, 3, H, D]
            qd, kd, vd = qkv[:, :, 0], qkv[:, :, 1], qkv[:, :, 2]
        else:
            qd, kd, vd = dev(q), dev(k), dev(v)
        qr = self.lib.unstep_kv_append_qknorm(f0, C, qd if with_q else None, kd, vd, cos_t, sin_t,
                                              dev(wq_bits) if with_q else None, dev(wk_bits), eps)
        c, s = tables.rope_tables(f0, C, self.gh, self.gw)
        shape = k.shape
        flat = shape[:-2] + (shape[-2] * shape[-1],)
        kn = rmsnorm.rms_norm_bf16(k.reshape(flat), wk_bits, eps).reshape(shape)
        self.orc.append(f0, C, rope.rope_bf16(kn, c, s), v)
        if not with_q:
            return None, None
        qn = rmsnorm.rms_norm_bf16(q.reshape(flat), wq_bits, eps).reshape(shape)
        return qr, rope.rope_bf16(qn, c, s)

    def step(self, f0: int, C: int, W: int, key, use_split=True, lse=False, q_layout="contiguous", **kw):
        """One whole chunk step through unstep_step; returns (q_rot_dev, out_dev, lse_dev, q_rot_oracle)."""
        q, k, v = self.inputs(C, key, **kw)
        cos_t, sin_t = self.tables.get(f0, C, self.gh, self.gw)
        if q_layout == "fused_qkv":
            qkv = torch.stack([dev(q), dev(k), dev(v)], dim=2)       # [B, N, 3, H, D]
            qd, kd, vd = qkv[:, :, 0], qkv[:, :, 1], qkv[:, :, 2]
        else:
            qd, kd, vd = dev(q), dev(k), dev(v)
        lse_t = torch.empty((self.B, self.H, C * self.T), dtype=torch.float32, device=qd.device) if lse else None
        q_rot = torch.empty((self.B, C * self.T, self.H, 128), dtype=torch.bfloat16, device=qd.device)
        out = self.lib.unstep_step(f0, C, W, qd, kd, vd, cos_t, sin_t, q_rot=q_rot, lse=lse_t, use_split=use_split)
        c, s = tables.rope_tables(f0, C, self.gh, self.gw)
        self.orc.append(f0, C, rope.rope_bf16(k, c, s), v)
        return q_rot, out, lse_t, rope.rope_bf16(q, c, s)

    def check_cache(self, what: str) -> None:
        fm, newest = self.lib.frame_map()
        assert fm == self.orc.frame_of_slot and newest == self.orc.newest, what
        assert np.array_equal(host(self.lib.k), self.orc.k), f"{what}: K cache differs"
        assert np.array_equal(host(self.lib.v), self.orc.v), f"{what}: V cache differs"
        if self.guard:
            g = self.guard
            n = self.B * self.H * self.slots
            for full, val in ((self.k_full, 1.5), (self.v_full, -2.5)):
                assert bool((full[:g] == val).all()) and bool((full[g + n:] == val).all()), f"{what}: guard band"

    def expected(self, q_rot_bits, f0, C, W, query_idx=None, heads=None):
        rows = self.orc.key_rows(f0, C, W)
        return attention.attention(q_rot_bits, self.orc.k, self.orc.v, rows, query_idx=query_idx, heads=heads)


def sample_queries(N: int, n: int, seed: int) -> np.ndarray:
    """A sorted random subset of query rows, always including the first and last."""
    rng = np.random.default_rng(seed)
    idx = set(rng.choice(N, size=min(n, N), replace=False).tolist()) | {0, N - 1}
    return np.array(sorted(idx), dtype=np.int64)


def random_shape_cases(n_cases: int = 48, seed: int = 2609) -> list:
    """Seeded small configurations for the randomized parity test: batch 1-2, 1-4 heads, grids
    up to 8x12 (ragged query and key tiles; the second case has one token per frame), 0-2 sinks (chunks that straddle the
    sink boundary), chunks of 1-3 frames, windows of 0-9 frames and rings up to 2 frames larger
    than they need.  Each case carries a call sequence of in-order chunks with repeats of the
    newest chunk, each call on the balanced or the plain schedule, with or without LSE."""
    rng = np.random.default_rng([seed, 7])
    cases = []
    for i in range(n_cases):
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 5))
        gh, gw = int(rng.integers(1, 9)), int(rng.integers(1, 13))
        if i == 1:
            gh = gw = 1                                     # one token per frame
        S, C, W = int(rng.integers(0, 3)), int(rng.integers(1, 4)), int(rng.integers(0, 10))
        R = W + C + int(rng.integers(0, 3))
        calls, f0 = [], 0
        for _ in range(int(rng.integers(6, 12))):
            calls.append((f0, bool(rng.integers(0, 4) > 0), bool(rng.integers(0, 2))))
            if rng.random() < 0.75:
                f0 += C
        cases.append(dict(B=B, H=H, gh=gh, gw=gw, S=S, R=R, C=C, W=W, calls=calls))
    return cases


def random_medium_cases(n_cases: int = 16, seed: int = 4242) -> list:
    """Seeded medium configurations: grids 4x4 to 16x16, 1-6 heads, up to 3 sinks and 12-frame
    windows, so walks run over tens of key tiles, through several runs of a wrapped ring and
    on every schedule (one work-group per query tile, the balanced split, the equal split of
    each query tile); call sequences as in random_shape_cases."""
    rng = np.random.default_rng([seed, 9])
    cases = []
    for _ in range(n_cases):
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 7))
        gh, gw = int(rng.integers(4, 17)), int(rng.integers(4, 17))
        S, C, W = int(rng.integers(0, 4)), int(rng.integers(1, 4)), int(rng.integers(0, 13))
        R = W + C + int(rng.integers(0, 3))
        calls, f0 = [], 0
        for _ in range(int(rng.integers(4, 9))):
            calls.append((f0, bool(rng.integers(0, 4) > 0), bool(rng.integers(0, 2))))
            if rng.random() < 0.8:
                f0 += C
        cases.append(dict(B=B, H=H, gh=gh, gw=gw, S=S, R=R, C=C, W=W, calls=calls))
    return cases
