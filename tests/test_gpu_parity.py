"""GPU parity of the chunk step against the oracle, through the C ABI.

Bar: q_rot, the K/V cache buffers and the host index state bit-exact; attention
within max-abs 2e-2 and mean-abs 2e-3 (bf16 inputs, fp32 accumulation) plus a
relative mean bound (gpu_helpers).  The workloads are the five named shapes
(tiny; full-frame chunk; unwindowed; short window + refine over 30 layers;
60-chunk rolling stream), the paper's own 3-sink window, and edge cases: a
ragged odd grid with batch 2 and sinks, fused-QKV strides, guard bands, closed-form
probes (Q = 0, V = 1, needle key), peaky softmax, and split vs unsplit keys.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import numerics
from tests.gpu_helpers import LSE_ABS, Mirror, check_attention, dev, host, log, sample_queries

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def u():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32518_amd as lib
    return lib


def _prefill(m: Mirror, wl, key0, upto: int, keep_from: int = 0):
    """Frames [0, upto) in chunks of wl.C: frames before keep_from are recorded without
    data (evicted before use), later ones appended with random K/V."""
    for f0 in range(0, upto, wl.C):
        C = min(wl.C, upto - f0)
        if f0 + C <= keep_from:
            m.skip_frames(f0, C)
        else:
            m.append(f0, C, (key0 if isinstance(key0, tuple) else (key0,)) + (f0,))


def test_tiny_full_compare(u):
    wl = synth.WORKLOADS["tiny"]
    log("tiny: B=1 H=2 grid 4x6 chunk@6 W=6")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R, guard_rows=64)
    _prefill(m, wl, 1, wl.f0)
    q_rot, out, lse, q_rot_ref = m.step(wl.f0, wl.C, wl.W, (1, 100), lse=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(q_rot), q_rot_ref)
    m.check_cache("tiny")
    want, want_lse = m.expected(q_rot_ref, wl.f0, wl.C, wl.W)
    log(f"  {check_attention(host(out), want, 'tiny')}")
    assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS


@pytest.mark.parametrize("use_split", [True, False])
def test_full_chunk(u, use_split):
    wl = synth.WORKLOADS["full_chunk"]
    log(f"full_chunk: H=12 30x52 chunk@9 W=9 split={use_split}")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    _prefill(m, wl, 2, wl.f0)
    q_rot, out, lse, q_rot_ref = m.step(wl.f0, wl.C, wl.W, (2, 100), use_split=use_split, lse=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(q_rot), q_rot_ref)
    m.check_cache("full_chunk")
    assert m.lib.segments(wl.f0, wl.C, wl.W) == [(0, 18720)]
    # every query x head x dim against the oracle
    want, want_lse = m.expected(q_rot_ref, wl.f0, wl.C, wl.W)
    log(f"  {check_attention(host(out), want, 'full_chunk')}")
    assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS


def test_unwindowed(u):
    wl = synth.WORKLOADS["unwindowed"]
    log("unwindowed: chunk@18 W=18 (32760 keys)")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    _prefill(m, wl, 3, wl.f0)
    # the balanced schedule: the merge kernel writes both the output and the log-sum-exp
    assert m.lib.workspace_bytes(wl.f0, wl.C, wl.W) > 0
    q_rot, out, lse, q_rot_ref = m.step(wl.f0, wl.C, wl.W, (3, 100), lse=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(q_rot), q_rot_ref)
    m.check_cache("unwindowed")
    want, want_lse = m.expected(q_rot_ref, wl.f0, wl.C, wl.W)
    log(f"  {check_attention(host(out), want, 'unwindowed')}")
    assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS


@pytest.mark.parametrize("group", [0, 1, 2])
def test_short_window_refine_30_layers(u, group):
    wl = synth.WORKLOADS["short_refine"]
    log(f"short_refine: layers {10 * group}..{10 * group + 9} of 30, 2 passes, chunk@12 W=3 R=6 (wraps)")
    for layer in range(10 * group, 10 * group + 10):
        m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
        # frames 0..8 are evicted before the chunk at 12 reads the cache; 9..11 are the window
        _prefill(m, wl, (4, layer), wl.f0, keep_from=wl.f0 - wl.W)
        for p in range(wl.passes):
            q_rot, out, _, q_rot_ref = m.step(wl.f0, wl.C, wl.W, (4, layer, 100, p))
            torch.cuda.synchronize()
            assert np.array_equal(host(q_rot), q_rot_ref)
            if layer % 10 == 0 or p == wl.passes - 1:
                m.check_cache(f"short_refine layer {layer} pass {p}")
            # every query of one head per call (all heads in the first layer of each group)
            heads = list(range(wl.H)) if layer % 10 == 0 else [layer % 12]
            want, _ = m.expected(q_rot_ref, wl.f0, wl.C, wl.W, heads=heads)
            got = host(out)[:, :, heads]
            st = check_attention(got, want, f"short_refine layer {layer} pass {p}")
        assert m.lib.segments(wl.f0, wl.C, wl.W) == [(3 * 1560, 3 * 1560), (0, 3 * 1560)]
        if layer % 10 == 0:
            log(f"  layer {layer}: {st}")


def test_rolling_stream_60_chunks(u):
    wl = synth.WORKLOADS["rolling"]
    log("rolling: 60 one-frame chunks through a 12-frame ring")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    for c in range(wl.chunks):
        with_lse = c % 5 == 4          # the equal split of each query tile and its merge, with LSE
        q_rot, out, lse, q_rot_ref = m.step(c, 1, wl.W, (5, c), lse=with_lse)
        torch.cuda.synchronize()
        assert np.array_equal(host(q_rot), q_rot_ref), c
        m.check_cache(f"rolling chunk {c}")
        # every query at the empty start, the first full window, the first wrap and the end;
        # a sample of rows elsewhere
        idx = np.arange(wl.n_query) if c in (0, 11, 12, 59) else sample_queries(wl.n_query, 24, 100 + c)
        want, want_lse = m.expected(q_rot_ref, c, 1, wl.W, query_idx=idx)
        st = check_attention(host(out)[:, idx], want, f"rolling chunk {c}")
        if with_lse:
            assert np.max(np.abs(lse.cpu().numpy()[:, :, idx] - want_lse)) <= LSE_ABS, c
        if c % 15 == 0 or c == wl.chunks - 1:
            log(f"  chunk {c}: keys {min(c + 1, 12) * 1560} {st}")


def test_paper_default_sinks(u):
    wl = synth.WORKLOADS["paper_default"]
    log("paper_default: 3 sinks + 6 recent frames (14040 keys)")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    _prefill(m, wl, 6, wl.f0)
    q_rot, out, lse, q_rot_ref = m.step(wl.f0, wl.C, wl.W, (6, 100), lse=True)
    torch.cuda.synchronize()
    assert np.array_equal(host(q_rot), q_rot_ref)
    m.check_cache("paper_default")
    assert sum(l for _, l in m.lib.segments(wl.f0, wl.C, wl.W)) == 14040
    want, want_lse = m.expected(q_rot_ref, wl.f0, wl.C, wl.W)
    assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS
    log(f"  {check_attention(host(out), want, 'paper_default')}")


# Exact-max re-walk.  The kernel fixes each row's exponent offset at the maximum of the first
# key tile of its range; a row whose scores later exceed that offset by more than
# 64 / (scale log2 e) ~ 502 raw units overflows the 2^64 row-sum guard, and the work-group
# walks its range again, first for the exact row maximum, then for the sums.  Here one head
# gets needle keys: raw keys drawn N(0, 40^2) at several tokens of the chunk (the end of the
# key range), so that about one query in eight scores more than 530 on them.  Run at the
# full-frame shape on the plain schedule (one work-group per query tile, a single run of
# cache rows), at the unwindowed shape on both schedules, and on a wrapped window whose rows
# form two runs (the loader's multi-run path); every element against the oracle.
# A six-frame window at frame 27 of a twelve-frame ring: frames 21-29 sit in slots 9-11 and 0-5,
# two runs of cache rows even in cache order, so the loader takes its multi-run path.
WRAPPED_WINDOW = synth.Workload("wrapped_window", B=1, H=12, D=128, grid_h=30, grid_w=52, C=3, S=0, W=6, R=12,
                                f0=27)


@pytest.mark.parametrize("workload,use_split", [("full_chunk", False), ("unwindowed", True),
                                                ("unwindowed", False), ("wrapped_window", False)])
def test_exact_max_rewalk(u, workload, use_split):
    wl = WRAPPED_WINDOW if workload == "wrapped_window" else synth.WORKLOADS[workload]
    log(f"rewalk: {workload} split={use_split}, needle keys in head 0")
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    _prefill(m, wl, 17, wl.f0, keep_from=wl.f0 - wl.W)
    if use_split:
        assert m.lib.workspace_bytes(wl.f0, wl.C, wl.W) > 0
    key = (17, 100)
    shape = (wl.B, wl.n_query, wl.H, 128)
    k = synth.normal_bf16(shape, key + (synth.K,))
    needles = [100, 1100, 2100, 3100, 4100]
    for j, t in enumerate(needles):
        k[0, t, 0] = synth.normal_bf16((128,), key + (50 + j,), scale=40.0)
    q_rot, out, lse, q_rot_ref = m.step(wl.f0, wl.C, wl.W, key, use_split=use_split, lse=True, k_bits=k)
    torch.cuda.synchronize()
    assert np.array_equal(host(q_rot), q_rot_ref)
    m.check_cache(f"rewalk {workload}")
    if workload == "wrapped_window":
        assert m.lib.segments(wl.f0, wl.C, wl.W) == [(9 * wl.T, 3 * wl.T), (0, 6 * wl.T)]
    # the construction does trigger the guard: some row of head 0 scores more than 502 raw units
    # above the maximum of its first key tile (the launch walks the retained rows in ascending
    # cache order and, on the plain schedule, from the first of them)
    rows = m.orc.key_rows(wl.f0, wl.C, wl.W)
    qh = numerics.bf16_to_f64(q_rot_ref[0, :, 0])
    s_first = qh @ numerics.bf16_to_f64(m.orc.k[0, 0, np.sort(rows)[:64]]).T
    s_needle = qh @ numerics.bf16_to_f64(m.orc.k[0, 0, rows[-wl.n_query:][needles]]).T
    jump = s_needle.max(axis=1) - s_first.max(axis=1)
    log(f"  rows past the guard: {int((jump > 64 / (128 ** -0.5 * math.log2(math.e))).sum())} of {wl.n_query}")
    assert (jump > 530).sum() > wl.n_query // 20
    want, want_lse = m.expected(q_rot_ref, wl.f0, wl.C, wl.W)
    log(f"  {check_attention(host(out), want, 'rewalk ' + workload)}")
    assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS


@pytest.mark.parametrize("use_split", [True, False])
def test_ragged_batch2_sinks_fused_qkv(u, use_split):
    # 5x7 grid (35 tokens/frame: ragged query and key tiles), batch 2, 3 heads, 2 sinks,
    # 16-frame ring with 2-frame chunks and a 13-frame window (wraps; up to 595 keys, enough
    # tiles for the key range to be split), fused [B, N, 3, H, D] input strides, guard bands
    log(f"ragged: B=2 H=3 grid 5x7 S=2 R=16 C=2 W=13 split={use_split}")
    m = Mirror(u, 2, 3, 5, 7, 2, 16, guard_rows=128)
    for ci, f0 in enumerate(range(0, 40, 2)):
        if ci == 12:
            assert m.lib.workspace_bytes(f0, 2, 13) > 0      # this shape takes the split path
        q_rot, out, lse, q_rot_ref = m.step(f0, 2, 13, (7, ci), use_split=use_split, lse=True,
                                            q_layout="fused_qkv" if ci % 2 else "contiguous")
        torch.cuda.synchronize()
        assert np.array_equal(host(q_rot), q_rot_ref), f0
        m.check_cache(f"ragged chunk {f0}")
        want, want_lse = m.expected(q_rot_ref, f0, 2, 13)
        check_attention(host(out), want, f"ragged chunk {f0}")
        assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS


def test_refine_overwrites_in_place(u):
    wl = synth.WORKLOADS["tiny"]
    m = Mirror(u, wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    _prefill(m, wl, 11, 6)
    before = m.lib.frame_map()
    for p in range(3):
        m.step(6, 3, 6, (11, 100 + p))
    torch.cuda.synchronize()
    fm, newest = m.lib.frame_map()
    assert newest == 8 and fm[:9] == list(range(9))
    m.check_cache("refine overwrite")


def test_probe_zero_queries_mean_of_frame_values(u):
    # Q = 0 -> uniform softmax; V = frame index -> every output is the mean retained frame index
    S, R, W, C, gh, gw = 3, 6, 3, 3, 6, 10
    m = Mirror(u, 1, 2, gh, gw, S, R)
    T = gh * gw
    for ci, f0 in enumerate(range(0, 15, 3)):
        frames = f0 + np.arange(C * T) // T
        vb = synth.small_int_bf16((1, C * T, 2, 128), frames[None, :, None, None])
        q_rot, out, lse, _ = m.step(f0, C, W, (12, ci), q_zero=True, v_bits=vb, lse=True)
        torch.cuda.synchronize()
        lo = max(0, f0 - W)
        kept = list(range(min(S, lo))) + list(range(lo, f0 + C))
        want = np.float32(np.mean(kept))
        got = numerics.bf16_to_f64(host(out))
        assert np.max(np.abs(got - want)) <= abs(want) * 2.0 ** -8, (f0, want)
        assert np.max(np.abs(lse.cpu().numpy() - math.log(len(kept) * T))) < 1e-5


def test_probe_unit_values_rows_sum_to_one(u):
    m = Mirror(u, 1, 4, 8, 9, 0, 4)
    ones = synth.small_int_bf16((1, 2 * 72, 4, 128), np.ones(1))
    m.append(0, 2, (13, 0), v_bits=ones)
    q_rot, out, _, _ = m.step(2, 2, 2, (13, 1), v_bits=ones, q_scale=4.0)
    torch.cuda.synchronize()
    assert np.max(np.abs(numerics.bf16_to_f64(host(out)) - 1.0)) <= 2.0 ** -8


def test_probe_needle_key(u):
    # key 37 of frame 1 equals 6 x the query of token 0 (head 0): token 0's output is that key's V
    m = Mirror(u, 1, 2, 4, 6, 0, 6)
    q, k, v = m.inputs(3, (14, 0))
    c, s = m.tables.get(0, 3, 4, 6)
    from oracle import rope, tables as otab
    oc, os_ = otab.rope_tables(0, 3, 4, 6)
    q_rot_ref = rope.rope_bf16(q, oc, os_)
    # choose raw key so that after rotation it is close to 6 * q_rot[0]: rotate back exactly in fp64
    target = 6.0 * numerics.bf16_to_f64(q_rot_ref[0, 0, 0])
    ang = otab.angles_f64(0, 3, 4, 6, 128, 10000.0)[24 + 13]
    te, to = target[0::2], target[1::2]
    raw = np.empty(128)
    raw[0::2] = te * np.cos(ang) + to * np.sin(ang)
    raw[1::2] = -te * np.sin(ang) + to * np.cos(ang)
    k = k.copy()
    k[0, 24 + 13, 0] = synth.bf16_bits_from_f32(raw.astype(np.float32))
    qd, kd, vd = dev(q), dev(k), dev(v)
    out = m.lib.unstep_step(0, 3, 0, qd, kd, vd, c, s)
    torch.cuda.synchronize()
    m.orc.append(0, 3, rope.rope_bf16(k, oc, os_), v)
    want, _ = m.expected(q_rot_ref, 0, 3, 0, query_idx=[0], heads=[0])
    got = numerics.bf16_to_f64(host(out)[0, 0, 0])
    needle_v = numerics.bf16_to_f64(v[0, 24 + 13, 0])
    assert np.max(np.abs(want[0, 0, 0] - needle_v)) < 0.05        # the oracle agrees it is a needle
    assert np.max(np.abs(got - want[0, 0, 0])) < 2e-2


def test_peaky_softmax(u):
    wl = synth.WORKLOADS["tiny"]
    m = Mirror(u, 1, 2, 6, 8, 0, 9)
    _prefill(m, wl, 15, 6)
    q_rot, out, _, q_rot_ref = m.step(6, 3, 6, (15, 100), q_scale=8.0)
    torch.cuda.synchronize()
    want, _ = m.expected(q_rot_ref, 6, 3, 6)
    log(f"  peaky: {check_attention(host(out), want, 'peaky')}")


def test_separate_calls_equal_step(u):
    # unstep_kv_append + unstep_window_attn give the same bits as unstep_step
    wl = synth.WORKLOADS["tiny"]
    a = Mirror(u, 1, 2, 4, 6, 0, 9)
    b = Mirror(u, 1, 2, 4, 6, 0, 9)
    for mm in (a, b):
        _prefill(mm, wl, 16, 6)
    q_rot, out, _, _ = a.step(6, 3, 6, (16, 100))
    q, k, v = b.inputs(3, (16, 100))
    cos_t, sin_t = b.tables.get(6, 3, 4, 6)
    qr = b.lib.unstep_kv_append(6, 3, dev(q), dev(k), dev(v), cos_t, sin_t)
    out2 = b.lib.unstep_window_attn(6, 3, 6, qr)
    torch.cuda.synchronize()
    assert torch.equal(q_rot.view(torch.int16), qr.view(torch.int16))
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    assert torch.equal(a.lib.k.view(torch.int16), b.lib.k.view(torch.int16))


def test_device_tables_equal_host_tables(u):
    for args in ((9, 3, 30, 52), (59, 1, 30, 52), (6, 3, 4, 6)):
        c, s = u.unstep_rope_tables(*args)
        hc, hs = u.unstep_rope_tables_host(*args)
        assert np.array_equal(c.cpu().numpy().view(np.uint32), hc.view(np.uint32))
        assert np.array_equal(s.cpu().numpy().view(np.uint32), hs.view(np.uint32))
