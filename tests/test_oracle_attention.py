"""Pins for the oracle's windowed attention (paper Sections 3.1, 3.3; Appendix A.3).

The paper prints no attention values, so the oracle is pinned by:
* brute force: the streamed ring cache + retained-key attention equals a full
  masked softmax over the whole frame timeline (no ring, explicit mask);
* a library routine: torch's scaled_dot_product_attention in float64;
* closed forms: Q = 0 gives the mean of the retained V rows (exact rationals
  with V = frame index); a needle key picks out its value row; one key gives
  its value; softmax rows sum to 1;
* window >= cache equals full block-causal attention;
* splitting the keys in two and merging by log-sum-exp equals the whole.
"""
import math

import numpy as np
import torch

import synth
from oracle import attention, numerics, rope, tables
from oracle.kvcache import KVCacheOracle


def _stream(S, R, W, C, n_chunks, gh=2, gw=3, H=2, seed=7, v_fn=None, q_scale=1.0):
    """Run n_chunks chunks through the oracle cache; return per-chunk outputs and the
    timeline of every frame's rotated keys/values."""
    D = 128
    T = gh * gw
    cache = KVCacheOracle(1, H, D, gh, gw, S, R)
    timeline_k, timeline_v, outs = [], [], []
    for ci in range(n_chunks):
        f0 = ci * C
        shape = (1, C * T, H, D)
        q = synth.normal_bf16(shape, (seed, ci, synth.Q), scale=q_scale)
        k = synth.normal_bf16(shape, (seed, ci, synth.K))
        v = synth.normal_bf16(shape, (seed, ci, synth.V)) if v_fn is None else v_fn(f0, shape)
        c, s = tables.rope_tables(f0, C, gh, gw)
        qr, kr = rope.rope_bf16(q, c, s), rope.rope_bf16(k, c, s)
        cache.append(f0, C, kr, v)
        timeline_k.append(kr)
        timeline_v.append(v)
        rows = cache.key_rows(f0, C, W)
        o, lse = attention.attention(qr, cache.k, cache.v, rows)
        outs.append((f0, qr, o, lse, rows))
    return cache, np.concatenate(timeline_k, axis=1), np.concatenate(timeline_v, axis=1), outs, T


def test_stream_equals_masked_timeline_bruteforce():
    for (S, R, W, C) in ((0, 9, 6, 3), (2, 4, 2, 1), (3, 6, 3, 3), (1, 5, 3, 2)):
        cache, tk, tv, outs, T = _stream(S, R, W, C, n_chunks=6)
        for f0, qr, o, lse, rows in outs:
            for h in range(cache.H):
                q = numerics.bf16_to_f64(qr[0, :, h, :])
                ref = attention.masked_timeline_attention(
                    q, f0, C, numerics.bf16_to_f64(tk[0, :, h, :]),
                    numerics.bf16_to_f64(tv[0, :, h, :]), T, S, W)
                assert np.max(np.abs(o[0, :, h, :] - ref)) < 1e-12


def test_window_at_least_cache_is_full_block_causal():
    # W larger than every prior frame: identical to attending over the whole prefix
    cache, tk, tv, outs, T = _stream(0, 12, 100, 3, n_chunks=4)
    for f0, qr, o, lse, rows in outs:
        assert rows.size == (f0 + 3) * T
        q = numerics.bf16_to_f64(qr[0, :, 0, :])
        K = numerics.bf16_to_f64(tk[0, :(f0 + 3) * T, 0, :])
        V = numerics.bf16_to_f64(tv[0, :(f0 + 3) * T, 0, :])
        p = attention.softmax_weights(q, K, 1 / math.sqrt(128))
        assert np.max(np.abs(o[0, :, 0, :] - p @ V)) < 1e-12


def test_matches_torch_sdpa_float64():
    cache, tk, tv, outs, T = _stream(3, 6, 3, 3, n_chunks=4)
    f0, qr, o, lse, rows = outs[-1]
    q = torch.from_numpy(numerics.bf16_to_f64(qr[0].transpose(1, 0, 2)))            # [H, N, D]
    k = torch.from_numpy(numerics.bf16_to_f64(cache.k[0][:, rows, :]))
    v = torch.from_numpy(numerics.bf16_to_f64(cache.v[0][:, rows, :]))
    ref = torch.nn.functional.scaled_dot_product_attention(q[None], k[None], v[None])[0]
    assert np.max(np.abs(o[0].transpose(1, 0, 2) - ref.numpy())) < 1e-12


def test_rows_sum_to_one_and_lse():
    rng = np.random.default_rng(3)
    q, K = rng.standard_normal((40, 128)), rng.standard_normal((300, 128))
    p = attention.softmax_weights(q, K, 1 / math.sqrt(128))
    assert np.max(np.abs(p.sum(axis=1) - 1.0)) < 1e-13
    s = (q @ K.T) / math.sqrt(128)
    lse_direct = np.log(np.exp(s).sum(axis=1))
    o, lse = attention._attend(q, K, rng.standard_normal((300, 128)), 1 / math.sqrt(128))
    assert np.max(np.abs(lse - lse_direct)) < 1e-12


def test_zero_queries_average_frame_index_values():
    # Q = 0: uniform softmax over retained keys; V = frame index (exact in bf16) =>
    # every output element equals the mean retained frame index, an exact rational.
    def v_fn(f0, shape):
        T = shape[1] // 3
        frames = f0 + np.arange(shape[1]) // T
        return synth.small_int_bf16(shape, frames[None, :, None, None])

    S, R, W, C = 3, 6, 3, 3
    cache, tk, tv, outs, T = _stream(S, R, W, C, n_chunks=5, v_fn=v_fn, q_scale=0.0)
    for f0, qr, o, lse, rows in outs:
        lo = max(0, f0 - W)
        frames = list(range(min(S, lo))) + list(range(lo, f0 + C))
        assert np.max(np.abs(o - np.mean(frames))) < 1e-12
        assert np.max(np.abs(lse - math.log(len(frames) * T))) < 1e-12


def test_needle_key_selects_its_value():
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 128))
    K = rng.standard_normal((500, 128))
    V = rng.standard_normal((500, 128))
    K[123] = 40.0 * q[0]
    o, _ = attention._attend(q, K, V, 1 / math.sqrt(128))
    assert np.max(np.abs(o[0] - V[123])) < 1e-9


def test_single_key_returns_its_value():
    rng = np.random.default_rng(12)
    o, lse = attention._attend(rng.standard_normal((5, 128)), rng.standard_normal((1, 128)),
                               np.arange(128.0)[None, :], 0.1)
    assert np.array_equal(o, np.tile(np.arange(128.0), (5, 1)))


def test_lse_split_merge_equals_whole():
    rng = np.random.default_rng(13)
    q, K, V = rng.standard_normal((64, 128)), rng.standard_normal((900, 128)), rng.standard_normal((900, 128))
    whole, _ = attention._attend(q, K, V, 0.09)
    parts = [attention._attend(q, K[a:b], V[a:b], 0.09) for a, b in ((0, 250), (250, 777), (777, 900))]
    merged = attention.merge_partials([p[0] for p in parts], [p[1] for p in parts])
    assert np.max(np.abs(merged - whole)) < 1e-13


def test_query_subset_and_head_subset_agree_with_full():
    cache, tk, tv, outs, T = _stream(0, 9, 6, 3, n_chunks=3)
    f0, qr, o, lse, rows = outs[-1]
    sel = [0, 5, 17]
    o2, l2 = attention.attention(qr, cache.k, cache.v, rows, query_idx=sel, heads=[1])
    assert np.array_equal(o2[0, :, 0, :], o[0, sel, 1, :])
    assert np.array_equal(l2[0, 0], lse[0, 1, sel])
