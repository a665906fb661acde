"""The C ABI library on the host, without a GPU: it loads, exports every symbol the
header declares, builds rotary tables bit-identical to the oracle's, keeps the same
host index state as the oracle's cache model, and rejects bad calls before touching
the device.  No kernel runs here.
"""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import synth
from oracle import tables
from oracle.kvcache import KVCacheOracle, OracleError

u = pytest.importorskip("paper_2609_32518_amd")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KIND = {"shape": u.E_SHAPE, "range": u.E_RANGE, "state": u.E_STATE, "null": u.E_NULL}

# fake, 16-byte aligned "device" addresses: host-only calls never dereference them
FAKE = [0x10000 * (i + 1) for i in range(12)]


def header_functions():
    text = open(os.path.join(ROOT, "include", "unstep.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(unstep_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = header_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(u.lib, n), n
    assert set(names) == set(u.SIGNATURES)


def test_version_and_error_string():
    assert u.version() == 100
    assert isinstance(u.lib.unstep_last_error(), bytes)


@pytest.mark.parametrize("args", [(9, 3, 30, 52), (6, 3, 4, 6), (0, 1, 1, 1), (59, 1, 30, 52), (123, 3, 5, 7),
                                  (18, 3, 30, 52)])
def test_host_tables_bit_identical_to_oracle(args):
    c, s = u.unstep_rope_tables_host(*args)
    oc, os_ = tables.rope_tables(*args)
    assert np.array_equal(c.view(np.uint32), oc.view(np.uint32))
    assert np.array_equal(s.view(np.uint32), os_.view(np.uint32))


def test_tables_argument_errors():
    buf = np.empty((100, 64), np.float32)
    p = buf.ctypes.data_as(u._pf32)
    assert u.lib.unstep_rope_tables_host(0, 1, 2, 2, 64, 10000.0, p, p) == u.E_SHAPE
    assert u.lib.unstep_rope_tables_host(0, 0, 2, 2, 128, 10000.0, p, p) == u.E_SHAPE
    assert u.lib.unstep_rope_tables_host(-1, 1, 2, 2, 128, 10000.0, p, p) == u.E_RANGE
    assert u.lib.unstep_rope_tables_host(0, 1, 2, 2, 128, 1.0, p, p) == u.E_RANGE
    assert u.lib.unstep_rope_tables_host(0, 1, 2, 2, 128, 10000.0, None, p) == u.E_NULL


def _handle(B, H, gh, gw, S, R, head_dim=128, k=FAKE[0], v=FAKE[1]):
    h = u._vp()
    rc = u.lib.unstep_cache_create(ctypes.byref(h), B, H, head_dim, gh, gw, S, R, k, v)
    return rc, h


def test_create_errors():
    assert _handle(1, 2, 2, 3, 0, 4, head_dim=64)[0] == u.E_SHAPE
    assert _handle(0, 2, 2, 3, 0, 4)[0] == u.E_SHAPE
    assert _handle(1, 2, 2, 3, -1, 4)[0] == u.E_SHAPE
    assert _handle(1, 2, 2, 3, 0, 0)[0] == u.E_SHAPE
    assert _handle(1, 2, 2, 3, 0, 4, k=0)[0] == u.E_NULL
    assert _handle(1, 2, 2, 3, 0, 4, k=FAKE[0] + 8)[0] == u.E_ALIGN
    # size limits: 2^31 bytes per (batch, head), 65535 (batch, head) pairs, and the append
    # pass's 32-bit piece count per frame (T * H * 16)
    assert _handle(1, 1, 4096, 2048, 0, 1)[0] == u.E_SHAPE                # 2^23 rows
    assert _handle(256, 256, 1, 1, 0, 1)[0] == u.E_SHAPE
    assert _handle(1, 64, 2048, 1024, 0, 1)[0] == u.E_SHAPE               # 2^21 tokens x 64 heads
    rc, h = _handle(1, 63, 2048, 1024, 0, 1)                              # 2^21 x 63 x 16 < 2^31
    assert rc == u.OK
    u.lib.unstep_cache_destroy(h)
    assert u.lib.unstep_cache_destroy(None) == u.OK


def _frame_map(h, n):
    fm = (ctypes.c_int32 * n)()
    nw = ctypes.c_int32()
    assert u.lib.unstep_cache_frame_map(h, fm, ctypes.byref(nw)) == u.OK
    return list(fm), nw.value


def _segments(h, f0, C, W):
    r0 = (ctypes.c_int32 * 4)()
    ln = (ctypes.c_int32 * 4)()
    n = ctypes.c_int32()
    rc = u.lib.unstep_window_segments(h, f0, C, W, r0, ln, ctypes.byref(n))
    return rc, [(r0[i], ln[i]) for i in range(n.value)] if rc == u.OK else None


def _oracle_call(fn):
    try:
        return u.OK, fn()
    except OracleError as e:
        return KIND[e.kind], None


@pytest.mark.parametrize("S,R,C,W", [(0, 9, 3, 6), (3, 6, 3, 3), (0, 12, 1, 11), (2, 4, 1, 2), (1, 5, 2, 3),
                                     (0, 21, 3, 18), (0, 6, 3, 3)])
def test_index_state_matches_oracle_over_a_random_call_sequence(S, R, C, W):
    # random mix of in-order appends, repeated (refine) appends, older re-appends, gaps and
    # window queries; the library's status, frame map and segments must equal the oracle's
    gh, gw = 2, 3
    rc, h = _handle(1, 1, gh, gw, S, R)
    assert rc == u.OK
    orc = KVCacheOracle(1, 1, 128, gh, gw, S, R)
    rng = np.random.default_rng(S * 1000 + R * 100 + C * 10 + W)
    zeros = np.zeros((1, C * gh * gw, 1, 128), np.uint16)
    try:
        for step in range(300):
            op = rng.integers(0, 4)
            f0 = int(max(0, orc.newest + 1 + rng.integers(-2 * R, 3)))
            if op <= 1:
                code, _ = _oracle_call(lambda: orc.append(f0, C, zeros, zeros))
                assert u.lib.unstep_cache_advance(h, f0, C) == code, (step, f0)
            else:
                w = int(rng.integers(0, W + 3))
                code, segs = _oracle_call(lambda: orc.segments(f0, C, w))
                rc, got = _segments(h, f0, C, w)
                assert rc == code, (step, f0, w)
                if code == u.OK:
                    assert got == segs
                    rows = orc.key_rows(f0, C, w)
                    assert sum(l for _, l in got) == rows.size
            fm, newest = _frame_map(h, S + R)
            assert fm == orc.frame_of_slot and newest == orc.newest
    finally:
        u.lib.unstep_cache_destroy(h)


def test_paper_window_segments_and_key_counts():
    # 3 sinks + 6 recent frames including the chunk (14040 keys at 30x52), ring of 6
    rc, h = _handle(1, 12, 30, 52, 3, 6)
    for f0 in range(0, 12, 3):
        assert u.lib.unstep_cache_advance(h, f0, 3) == u.OK
    rc, segs = _segments(h, 9, 3, 3)
    assert rc == u.OK and sum(l for _, l in segs) == 14040
    assert segs == [(0, 3 * 1560), (6 * 1560, 3 * 1560), (3 * 1560, 3 * 1560)]
    u.lib.unstep_cache_destroy(h)


def test_append_errors_are_caught_before_any_device_work():
    rc, h = _handle(1, 2, 2, 3, 0, 4)
    T = 6
    p = FAKE
    args = lambda f0, C, q=None, qr=None, ts=256, hs=128, k=p[2]: (h, f0, C, q, k, p[3], ts, hs, p[4], p[5], qr, None)
    assert u.lib.unstep_kv_append(*args(1, 1)) == u.E_STATE              # gap
    assert u.lib.unstep_kv_append(*args(0, 0)) == u.E_SHAPE              # empty chunk
    assert u.lib.unstep_kv_append(*args(-1, 1)) == u.E_RANGE
    assert u.lib.unstep_kv_append(*args(0, 5)) == u.E_RANGE              # more than the ring
    assert u.lib.unstep_kv_append(*args(0, 1, k=None)) == u.E_NULL
    assert u.lib.unstep_kv_append(*args(0, 1, q=p[6])) == u.E_NULL       # q without q_rot
    assert u.lib.unstep_kv_append(*args(0, 1, ts=200)) == u.E_SHAPE      # tokens overlap
    assert u.lib.unstep_kv_append(*args(0, 1, ts=264, hs=132)) == u.E_ALIGN
    assert u.lib.unstep_kv_append(*args(0, 1, k=p[2] + 4)) == u.E_ALIGN
    assert u.lib.unstep_kv_append(None, 0, 1, None, p[2], p[3], 256, 128, p[4], p[5], None, None) == u.E_NULL
    assert _frame_map(h, 4) == ([-1] * 4, -1)
    # attention: nothing stored yet
    out = (h, 0, 1, 0, p[6], p[7], None, 0.0, None, 0, None)
    assert u.lib.unstep_window_attn(*out) == u.E_STATE
    assert u.lib.unstep_window_attn(h, 0, 1, 0, None, p[7], None, 0.0, None, 0, None) == u.E_NULL
    assert u.lib.unstep_cache_advance(h, 0, 3) == u.OK
    assert u.lib.unstep_window_attn(h, 3, 1, 3, p[6], p[7], None, 0.0, None, 0, None) == u.E_STATE
    assert u.lib.unstep_window_attn(h, 3, 2, 3, p[6], p[7], None, 0.0, None, 0, None) == u.E_RANGE  # 5 > 4 ring frames
    assert u.lib.unstep_window_attn(h, 2, 1, 2, p[6] + 2, p[7], None, 0.0, None, 0, None) == u.E_ALIGN
    # step: the attention half is checked on the post-append state, before anything runs
    st = lambda f0, C, W: u.lib.unstep_step(h, f0, C, W, p[6], p[2], p[3], 256, 128, p[4], p[5], p[8], p[9],
                                            None, 0.0, None, 0, None)
    assert st(3, 2, 3) == u.E_RANGE                                     # 3 prior + 2 > 4 ring frames
    assert st(5, 1, 1) == u.E_STATE                                     # gap
    assert _frame_map(h, 4) == ([0, 1, 2, -1], 2)
    u.lib.unstep_cache_destroy(h)


def test_qknorm_append_errors_are_caught_before_any_device_work():
    rc, h = _handle(1, 2, 2, 3, 0, 4)
    p = FAKE
    app = lambda f0=0, C=1, q=None, qr=None, wq=None, wk=p[10], eps=1e-6, k=p[2]: u.lib.unstep_kv_append_qknorm(
        h, f0, C, q, k, p[3], 256, 128, p[4], p[5], wq, wk, eps, qr, None)
    assert app(wk=None) == u.E_NULL                                     # k weight required
    assert app(q=p[6], qr=p[7], wq=None) == u.E_NULL                     # q without its weight
    assert app(eps=-1.0) == u.E_RANGE
    assert app(eps=float("inf")) == u.E_RANGE
    assert app(eps=float("nan")) == u.E_RANGE
    assert app(wk=p[10] + 8) == u.E_ALIGN
    assert app(f0=1) == u.E_STATE                                       # the append checks still apply
    assert app(k=None) == u.E_NULL
    assert _frame_map(h, 4) == ([-1] * 4, -1)
    u.lib.unstep_cache_destroy(h)
    rc, h33 = _handle(1, 33, 2, 3, 0, 4)                                # more heads than one wave holds
    assert rc == u.OK
    assert u.lib.unstep_kv_append_qknorm(h33, 0, 1, None, p[2], p[3], 33 * 128, 128, p[4], p[5], None, p[10], 1e-6,
                                         None, None) == u.E_SHAPE
    u.lib.unstep_cache_destroy(h33)


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-device error path")
def test_launch_failure_leaves_state_unchanged_without_a_device():
    rc, h = _handle(1, 2, 2, 3, 0, 4)
    p = FAKE
    rc = u.lib.unstep_kv_append(h, 0, 1, None, p[2], p[3], 256, 128, p[4], p[5], None, None)
    assert rc == u.E_HIP and u.lib.unstep_last_error()
    assert _frame_map(h, 4) == ([-1] * 4, -1)
    u.lib.unstep_cache_destroy(h)


def test_workspace_size_is_shape_only():
    rc, h = _handle(1, 12, 30, 52, 0, 12)
    b = ctypes.c_size_t()
    # nothing stored: the size query still answers (it depends on shapes only)
    assert u.lib.unstep_attn_workspace_size(h, 0, 1, 11, ctypes.byref(b)) == u.OK
    assert u.lib.unstep_attn_workspace_size(h, 0, 0, 11, ctypes.byref(b)) == u.E_SHAPE
    u.lib.unstep_cache_destroy(h)


def test_shift_schedule_bit_identical_to_oracle_and_errors():
    from oracle import schedule
    for n, shift in ((4, 5.0), (8, 3.0), (1, 5.0), (6, 1.0)):
        sigma, t = u.unstep_shift_schedule(n, shift)
        _, s_ref, t_ref = schedule.shift_schedule(n, shift)
        assert np.array_equal(sigma, s_ref) and np.array_equal(t, t_ref)
    d = ctypes.c_double()
    assert u.lib.unstep_shift_schedule(0, 5.0, ctypes.byref(d), ctypes.byref(d)) == u.E_SHAPE
    assert u.lib.unstep_shift_schedule(4, 0.0, ctypes.byref(d), ctypes.byref(d)) == u.E_RANGE
    assert u.lib.unstep_shift_schedule(4, 5.0, None, ctypes.byref(d)) == u.E_NULL


def test_renoise_emit_argument_errors():
    p = FAKE
    for fn in (u.lib.unstep_renoise, u.lib.unstep_emit):
        assert fn(None, p[1], 0.02, p[2], 100, None) == u.E_NULL
        assert fn(p[0], p[1], 0.02, p[2], -1, None) == u.E_SHAPE
        assert fn(p[0], p[1], 1.5, p[2], 100, None) == u.E_RANGE
        assert fn(p[0], p[1], float("nan"), p[2], 100, None) == u.E_RANGE
        assert fn(p[0] + 2, p[1], 0.02, p[2], 100, None) == u.E_ALIGN
        assert fn(p[0], p[1], 0.02, p[2], 0, None) == u.OK          # nothing to do


def test_sampler_calls_bit_identical_to_oracle_and_errors():
    from oracle import sampler
    for variant in sampler.VARIANTS:
        for n_chunks in (0, 1, 2, 7, 41):
            for cs in (None, 0.05):
                got = u.unstep_sampler_calls(variant, n_chunks, clean_sigma=cs)
                want = sampler.calls(variant, n_chunks, clean_sigma=cs)
                assert len(got["chunk"]) == len(want)
                for key, attr in (("chunk", "chunk"), ("start_frame", "start_frame"), ("schedule_index", "index"),
                                  ("sigma", "sigma"), ("t", "t")):
                    assert got[key].tolist() == [getattr(c, attr) for c in want], (variant, n_chunks, key)
    got = u.unstep_sampler_calls("unstep", 3, chunk_frames=1)
    assert got["start_frame"].tolist() == [c.start_frame for c in sampler.calls("unstep", 3, chunk_frames=1)]
    n = ctypes.c_int32(-7)
    i32 = ctypes.c_int32 * 8
    f64 = ctypes.c_double * 8
    a, b, c, d, e = i32(), i32(), i32(), f64(), f64()
    assert u.lib.unstep_sampler_calls(1, 2, 3, -1.0, 8, None, a, b, c, d, e) == u.E_NULL
    assert u.lib.unstep_sampler_calls(3, 2, 3, -1.0, 8, ctypes.byref(n), a, b, c, d, e) == u.E_RANGE
    assert u.lib.unstep_sampler_calls(1, -1, 3, -1.0, 8, ctypes.byref(n), a, b, c, d, e) == u.E_SHAPE
    assert u.lib.unstep_sampler_calls(1, 2, 0, -1.0, 8, ctypes.byref(n), a, b, c, d, e) == u.E_SHAPE
    assert u.lib.unstep_sampler_calls(1, 2, 3, 1.5, 8, ctypes.byref(n), a, b, c, d, e) == u.E_RANGE
    assert u.lib.unstep_sampler_calls(1, 2, 3, float("nan"), 8, ctypes.byref(n), a, b, c, d, e) == u.E_RANGE
    assert u.lib.unstep_sampler_calls(1, 2**30, 3, -1.0, 8, ctypes.byref(n), a, b, c, d, e) == u.E_RANGE
    # two chunks of the two-step sampler: 5 + 3 calls; capacity 7 is too small, the count is still reported
    assert u.lib.unstep_sampler_calls(1, 2, 3, -1.0, 7, ctypes.byref(n), a, b, c, d, e) == u.E_RANGE and n.value == 8
    assert u.lib.unstep_sampler_calls(1, 2, 3, -1.0, 8, ctypes.byref(n), a, None, c, d, e) == u.E_NULL
    assert u.lib.unstep_sampler_calls(1, 2, 3, -1.0, 8, ctypes.byref(n), a, b, c, d, e) == u.OK and n.value == 8
    assert u.lib.unstep_sampler_calls(1, 0, 3, -1.0, 0, ctypes.byref(n), None, None, None, None, None) == u.OK
    assert n.value == 0


def test_svd_and_linear_argument_errors():
    p = FAKE
    s = (ctypes.c_float * 4)()
    f = u.lib.unstep_svd_truncate
    assert f(None, 8, 8, 4, p[1], None, s, None) == u.E_NULL
    assert f(p[0], 8, 8, 4, None, None, s, None) == u.E_NULL
    assert f(p[0], 0, 8, 4, p[1], None, s, None) == u.E_SHAPE
    assert f(p[0], 1 << 15, 1 << 14, 4, p[1], None, s, None) == u.E_SHAPE
    assert f(p[0], 8, 6, 7, p[1], None, s, None) == u.E_RANGE
    assert f(p[0], 8, 6, -1, p[1], None, s, None) == u.E_RANGE
    assert f(p[0] + 4, 8, 8, 4, p[1], None, s, None) == u.E_ALIGN
    g = u.lib.unstep_linear
    assert g(None, p[1], None, p[2], 4, 8, 8, None) == u.E_NULL
    assert g(p[0], p[1], None, None, 4, 8, 8, None) == u.E_NULL
    assert g(p[0], p[1], None, p[2], 0, 8, 8, None) == u.E_SHAPE
    assert g(p[0], p[1], None, p[2], 4, 8, 12, None) == u.E_SHAPE
    assert g(p[0], p[1], None, p[2], 4, 12, 8, None) == u.E_SHAPE
    assert g(p[0], p[1], p[3] + 2, p[2], 4, 8, 8, None) == u.E_ALIGN


def test_schedule_choice_follows_the_measured_costs():
    # the attention plan (host arithmetic only): one work-group per query tile where the
    # balanced split over 256 compute units does not pay for its merge and its slower units
    # (the full-frame chunk, the paper's nine- and eight-frame windows, every call of a 5 s
    # clip), the balanced split where query tiles alone would leave many units idle (the
    # unwindowed 32,760-key call, one-frame rolling chunks)
    def ws(S, R, f0, C, W, H=12, gh=30, gw=52):
        rc, h = _handle(1, H, gh, gw, S, R)
        assert rc == u.OK
        b = ctypes.c_size_t(123)
        assert u.lib.unstep_attn_workspace_size(h, f0, C, W, ctypes.byref(b)) == u.OK
        u.lib.unstep_cache_destroy(h)
        return b.value
    assert ws(0, 12, 9, 3, 9) == 0                 # full-frame chunk, 18,720 keys
    assert ws(3, 6, 9, 3, 3) == 0                  # nine frames, 14,040 keys
    assert ws(2, 6, 9, 3, 3) == 0                  # eight frames
    assert ws(3, 6, 3, 3, 3) == 0                  # second chunk of a clip, six frames
    assert ws(0, 21, 18, 3, 18) > 0                # unwindowed, 32,760 keys
    assert ws(0, 12, 20, 1, 11) > 0                # one-frame chunk over 12 frames

    def part_bytes(groups):                          # two fp32 partials (o, offset, sum) per work-group
        return groups * 2 * 256 * (128 + 2) * 4
    # 84 query tiles: 3 work-groups per tile (252 of 256 units), each walks a third of a tile
    assert ws(0, 12, 20, 1, 11) == part_bytes(252)
    # 2 query tiles of 400 key tiles: 128 work-groups per tile would get 3 units each, so the
    # split stays at units / 4 = 200 (no work-group under 4 units, none empty)
    assert ws(0, 101, 100, 1, 99, H=2, gh=16, gw=16) == part_bytes(200)


def test_random_shape_cases_are_valid_and_reach_both_schedules():
    # the call sequences of the randomized GPU parity tests (small and medium shapes), replayed on
    # the host index and the oracle's cache model: every call is accepted by both with equal
    # segments, and the cases reach the plain schedule, the balanced one and its equal split of
    # each query tile, chunks across the sink boundary and single tokens
    from tests.gpu_helpers import random_medium_cases, random_shape_cases
    balanced = plain = straddle = equal_split = 0
    cases = random_shape_cases()
    for cs in cases + random_medium_cases():
        rc, h = _handle(cs["B"], cs["H"], cs["gh"], cs["gw"], cs["S"], cs["R"])
        assert rc == u.OK
        orc = KVCacheOracle(cs["B"], cs["H"], 128, cs["gh"], cs["gw"], cs["S"], cs["R"])
        C, W = cs["C"], cs["W"]
        zeros = np.zeros((cs["B"], C * cs["gh"] * cs["gw"], cs["H"], 128), np.uint16)
        try:
            for f0, use_split, _ in cs["calls"]:
                assert u.lib.unstep_cache_advance(h, f0, C) == u.OK
                orc.append(f0, C, zeros, zeros)
                rc, segs = _segments(h, f0, C, W)
                assert rc == u.OK and segs == orc.segments(f0, C, W)
                b = ctypes.c_size_t()
                assert u.lib.unstep_attn_workspace_size(h, f0, C, W, ctypes.byref(b)) == u.OK
                if use_split and b.value > 0:
                    balanced += 1
                    groups = b.value // (2 * 256 * (128 + 2) * 4)
                    qtiles = cs["B"] * cs["H"] * -(-C * cs["gh"] * cs["gw"] // 256)
                    equal_split += groups % qtiles == 0 and groups // qtiles >= 2
                else:
                    plain += 1
                straddle += f0 < cs["S"] < f0 + C
        finally:
            u.lib.unstep_cache_destroy(h)
    assert balanced >= 10 and plain >= 10 and straddle >= 2 and equal_split >= 5, (balanced, plain, straddle, equal_split)
    assert any(cs["gh"] * cs["gw"] == 1 for cs in cases)


def test_attention_rejects_more_query_tiles_than_one_launch_holds():
    # 255 x 256 (batch, head) pairs of 2-frame chunks of 32,768 tokens: 2^24 - 2^16 query tiles
    # of 256, more 512-thread work-groups than one launch dimension's 32-bit work-item count
    # holds; rejected before anything is enqueued
    rc, h = _handle(255, 256, 128, 256, 0, 2)
    assert rc == u.OK
    try:
        assert u.lib.unstep_cache_advance(h, 0, 2) == u.OK
        p = FAKE
        assert u.lib.unstep_window_attn(h, 0, 2, 0, p[6], p[7], None, 0.0, None, 0, None) == u.E_SHAPE
        assert b"query tiles" in u.lib.unstep_last_error()
        b = ctypes.c_size_t()
        assert u.lib.unstep_attn_workspace_size(h, 1, 1, 1, ctypes.byref(b)) == u.OK
    finally:
        u.lib.unstep_cache_destroy(h)


def test_binding_rejects_tensors_the_kernels_would_misread():
    # the library sees only pointers: the binding checks dtype, shape, device and layout of every
    # tensor against the handle before calling it (a CPU-side cache here: no call gets that far)
    B, H, gh, gw, S, R = 1, 2, 4, 6, 0, 9
    c = u.Cache(B, H, gh, gw, S, R, device="cpu")
    T, C = gh * gw, 3
    N = C * T
    bf = dict(dtype=torch.bfloat16)
    q = torch.zeros((B, N, H, 128), **bf)
    k, v = q.clone(), q.clone()
    cos_t = torch.zeros((N, 64), dtype=torch.float32)
    sin_t = cos_t.clone()
    bad = {
        "k dtype": dict(k=k.float()),
        "k tokens": dict(k=torch.zeros((B, N - 1, H, 128), **bf)),
        "k heads": dict(k=torch.zeros((B, N, H + 1, 128), **bf)),
        "k batch": dict(k=torch.zeros((B + 1, N, H, 128), **bf)),
        "k device": dict(k=torch.zeros((B, N, H, 128), device="meta", **bf)),
        "k last stride": dict(k=torch.zeros((B, N, 128, H), **bf).transpose(2, 3)),
        "v strides": dict(v=torch.zeros((B, N, 2, H, 128), **bf)[:, :, 0]),
        "cos rows": dict(cos_t=torch.zeros((N - 1, 64))),
        "sin dtype": dict(sin_t=torch.zeros((N, 64), dtype=torch.float64)),
        "q_rot shape": dict(q_rot=torch.zeros((B, N, H, 64), **bf)),
        "q_rot layout": dict(q_rot=torch.zeros((B, H, N, 128), **bf).transpose(1, 2)),
    }
    for what, kw in bad.items():
        args = dict(q=q, k=k, v=v, cos_t=cos_t, sin_t=sin_t, q_rot=None)
        args.update(kw)
        with pytest.raises(ValueError):
            c.unstep_kv_append(6, C, args["q"], args["k"], args["v"], args["cos_t"], args["sin_t"],
                               q_rot=args["q_rot"])
        with pytest.raises(ValueError):
            c.unstep_step(6, C, 6, args["q"], args["k"], args["v"], args["cos_t"], args["sin_t"],
                          q_rot=args["q_rot"])
    wn = torch.ones(H * 128, **bf)
    for kw in (dict(k_norm_weight=torch.ones(H * 128 - 8, **bf)), dict(q_norm_weight=torch.ones(H * 128)),
               dict(q_norm_weight=None)):
        args = dict(q_norm_weight=wn, k_norm_weight=wn)
        args.update(kw)
        with pytest.raises(ValueError):
            c.unstep_kv_append_qknorm(6, C, q, k, v, cos_t, sin_t, args["q_norm_weight"], args["k_norm_weight"])
    # attention: q_rot, out, lse
    for kw in (dict(q_rot=torch.zeros((B, N + 1, H, 128), **bf)),
               dict(q_rot=torch.zeros((B, H, N, 128), **bf).transpose(1, 2)),
               dict(out=torch.zeros((B, N, H, 128), dtype=torch.float16)),
               dict(out=torch.zeros((B, N, 128, H), **bf).transpose(2, 3)),
               dict(lse=torch.zeros((B, N, H))),
               dict(lse=torch.zeros((B, H, N), dtype=torch.float16))):
        args = dict(q_rot=q, out=None, lse=None)
        args.update(kw)
        with pytest.raises(ValueError):
            c.unstep_window_attn(6, C, 6, args["q_rot"], out=args["out"], lse=args["lse"])
        with pytest.raises(ValueError):
            c.unstep_step(6, C, 6, q, k, v, cos_t, sin_t, q_rot=args["q_rot"], out=args["out"], lse=args["lse"])
    # caller-given cache buffers of the wrong size or type
    with pytest.raises(ValueError):
        u.Cache(B, H, gh, gw, S, R, device="cpu", k_cache=torch.zeros((B, H, (S + R) * T - 1, 128), **bf))
    with pytest.raises(ValueError):
        u.Cache(B, H, gh, gw, S, R, device="cpu", v_cache=torch.zeros((B, H, (S + R) * T, 128)))
    # nothing was recorded by the rejected calls
    assert c.frame_map() == ([-1] * (S + R), -1)
    # clean-cache updates and the projection: shapes of caller outputs and devices
    x = torch.zeros((2, 8), **bf)
    with pytest.raises(ValueError):
        u.unstep_renoise(x, x, 0.1, out=torch.zeros((2, 16), **bf))
    with pytest.raises(ValueError):
        u.unstep_emit(x, torch.zeros((2, 8), device="meta", **bf), 0.1)
    with pytest.raises(ValueError):
        u.unstep_linear(torch.zeros((4, 8), **bf), torch.zeros((8, 8), **bf), out=torch.zeros((4, 16), **bf))


def test_huge_frame_requests_fail_fast_without_allocating():
    # a window or chunk of ~2^31 frames is rejected from the frame counts alone (no frame list
    # is built), so the call returns E_RANGE at once instead of exhausting host memory
    rc, h = _handle(1, 1, 2, 3, 2, 4)
    assert rc == u.OK
    try:
        assert u.lib.unstep_cache_advance(h, 0, 3) == u.OK
        big = 2_000_000_000
        assert _segments(h, big, 1, big)[0] == u.E_RANGE
        assert _segments(h, 0, big, 0)[0] == u.E_RANGE
        assert u.lib.unstep_cache_advance(h, 0, big) == u.E_RANGE
        ws = u._sz()
        assert u.lib.unstep_attn_workspace_size(h, big, 1, big, ctypes.byref(ws)) == u.E_RANGE
        assert u.lib.unstep_attn_workspace_size(h, 0, big, 0, ctypes.byref(ws)) == u.E_RANGE
        assert _frame_map(h, 6) == ([0, 1, 2, -1, -1, -1], 2)
    finally:
        u.lib.unstep_cache_destroy(h)


def test_noalloc_attention_checks_arguments_before_any_device_work():
    rc, h = _handle(1, 2, 4, 6, 0, 9)
    assert rc == u.OK
    try:
        f = u.lib.unstep_window_attn_noalloc
        assert f(None, 0, 1, 0, FAKE[2], FAKE[3], None, 0.0, None) == u.E_NULL
        assert f(h, 0, 1, 0, None, FAKE[3], None, 0.0, None) == u.E_NULL
        assert f(h, 0, 1, 0, FAKE[2], FAKE[3], None, 0.0, None) == u.E_STATE      # nothing appended
        assert u.lib.unstep_cache_advance(h, 0, 3) == u.OK
        assert f(h, 0, 3, 0, FAKE[2] + 8, FAKE[3], None, 0.0, None) == u.E_ALIGN
        assert f(h, 0, 3, 0, FAKE[2], FAKE[3], FAKE[4] + 2, 0.0, None) == u.E_ALIGN     # lse
        assert f(h, 5, 3, 0, FAKE[2], FAKE[3], None, 0.0, None) == u.E_STATE
    finally:
        u.lib.unstep_cache_destroy(h)


def test_mfma_reference_argument_errors():
    # every check runs before any device work: fake 16-byte aligned pointers are never touched
    f = u.lib.unstep_mfma_reference
    p = FAKE
    assert f(None, p[1], 4, 2, 64, None) == u.E_NULL
    assert f(p[0], None, 4, 2, 64, None) == u.E_NULL
    assert f(p[0], p[1], 0, 2, 64, None) == u.E_SHAPE
    assert f(p[0], p[1], 65537, 2, 64, None) == u.E_SHAPE
    assert f(p[0], p[1], 4, 0, 64, None) == u.E_SHAPE
    assert f(p[0], p[1], 4, 3, 64, None) == u.E_SHAPE
    assert f(p[0], p[1], 4, 2, 0, None) == u.E_SHAPE
    assert f(p[0], p[1], 4, 2, 48, None) == u.E_SHAPE
    assert f(p[0] + 8, p[1], 4, 2, 64, None) == u.E_ALIGN


def test_copy_reference_argument_errors():
    f = u.lib.unstep_copy3
    p = FAKE
    assert f(None, p[1], p[2], p[3], p[4], p[5], 64, None) == u.E_NULL
    assert f(p[0], p[1], p[2], p[3], p[4], None, 64, None) == u.E_NULL
    assert f(p[0], p[1], p[2], p[3], p[4], p[5], 60, None) == u.E_SHAPE
    assert f(p[0], p[1], p[2], p[3], p[4], p[5], -16, None) == u.E_SHAPE
    assert f(p[0] + 8, p[1], p[2], p[3], p[4], p[5], 64, None) == u.E_ALIGN
    assert f(p[0], p[1], p[2], p[3], p[4], p[5], 0, None) == u.OK          # nothing to copy, nothing launched
