"""Softmax attention of a chunk's queries over its retained keys (paper Sections 3.1
and 3.3; Appendix A.3 and A.5).

The windowed step is exact attention over a smaller key set, so the oracle is
the definition written out in float64:

    s_m = <q, k_m> * scale        scale = 1/sqrt(D) unless given
    p_m = exp(s_m - max s) / sum exp(s - max s)
    o   = sum_m p_m v_m,          lse = max s + log(sum exp(s - max s))

q, k, v are the bf16 values (exact in float64).  Matrix products use NumPy's
float64 matmul as a library primitive; rows are processed in blocks only to
bound memory, which does not change any value beyond float64 rounding order.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple

import numpy as np

from .numerics import bf16_to_f64


def _attend(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    s = (Q @ K.T) * scale
    m = s.max(axis=1)
    p = np.exp(s - m[:, None])
    l = p.sum(axis=1)
    o = (p @ V) / l[:, None]
    return o, m + np.log(l)


def attention(q_bits: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray, rows: np.ndarray,
              scale: Optional[float] = None, query_idx: Optional[Sequence[int]] = None,
              heads: Optional[Sequence[int]] = None, block: int = 512) -> Tuple[np.ndarray, np.ndarray]:
    """Attention of queries q[B, N, H, D] (bf16 bits) over cache rows `rows`.

    k_cache, v_cache: bf16 bits [B, H, slots, D]; rows: physical rows of the
    retained keys.  query_idx selects a subset of the N queries (default all),
    heads a subset of heads (default all).  Returns (o [B, n_sel, H_sel, D]
    float64, lse [B, H_sel, n_sel] float64, natural log).
    """
    B, N, H, D = q_bits.shape
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    qi = np.arange(N) if query_idx is None else np.asarray(query_idx, dtype=np.int64)
    hs = list(range(H)) if heads is None else list(heads)
    rows = np.asarray(rows, dtype=np.int64)
    o = np.empty((B, qi.size, len(hs), D), dtype=np.float64)
    lse = np.empty((B, len(hs), qi.size), dtype=np.float64)
    for b in range(B):
        for hi, h in enumerate(hs):
            K = bf16_to_f64(k_cache[b, h, rows, :])
            V = bf16_to_f64(v_cache[b, h, rows, :])
            for s0 in range(0, qi.size, block):
                sel = qi[s0:s0 + block]
                Q = bf16_to_f64(q_bits[b, sel, h, :])
                ob, lb = _attend(Q, K, V, scale)
                o[b, s0:s0 + sel.size, hi, :] = ob
                lse[b, hi, s0:s0 + sel.size] = lb
    return o, lse


def softmax_weights(q: np.ndarray, K: np.ndarray, scale: float) -> np.ndarray:
    """Softmax probabilities [n, M] of float64 queries q[n, D] over keys K[M, D]."""
    s = (q @ K.T) * scale
    p = np.exp(s - s.max(axis=1, keepdims=True))
    return p / p.sum(axis=1, keepdims=True)


def masked_timeline_attention(q: np.ndarray, q_frame_start: int, C: int, k_all: np.ndarray,
                              v_all: np.ndarray, T: int, S: int, W: int,
                              scale: Optional[float] = None) -> np.ndarray:
    """Brute-force reference over the whole frame timeline with an explicit mask.

    q: float64 [n, D] queries of the chunk starting at q_frame_start; k_all,
    v_all: float64 [F*T, D] keys/values of every frame 0..F-1 in time order (no
    ring buffer).  Key token j (frame j // T) is visible iff it is not in a
    later chunk (frame < q_frame_start + C) and it is either inside the window
    (frame >= q_frame_start - W) or a sink (frame < S).  Full softmax over the
    timeline with masked scores set to -inf.
    """
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[1])
    frame = np.arange(k_all.shape[0]) // T
    visible = (frame < q_frame_start + C) & ((frame >= q_frame_start - W) | (frame < S))
    s = (q @ k_all.T) * scale
    s = np.where(visible[None, :], s, -np.inf)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p = p / p.sum(axis=1, keepdims=True)
    return p @ v_all


def merge_partials(o_parts: Sequence[np.ndarray], lse_parts: Sequence[np.ndarray]) -> np.ndarray:
    """Combine attention results over disjoint key subsets by their log-sum-exp.

    o_parts[i]: [n, D] normalised outputs over subset i; lse_parts[i]: [n].
    The whole is sum_i exp(lse_i - lse) o_i with lse = log sum_i exp(lse_i).
    """
    L = np.stack(lse_parts)                      # [P, n]
    top = L.max(axis=0)
    w = np.exp(L - top)
    total = w.sum(axis=0)
    acc = sum(w[i][:, None] * o_parts[i] for i in range(len(o_parts)))
    return acc / total[:, None]
