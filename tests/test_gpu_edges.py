"""GPU edge cases of the chunk step through the C ABI: a single token attending to a single
key, a zero window with sinks, and a cache at the maximum size the ABI accepts (just under
2^31 bytes per (batch, head) buffer) whose ring has wrapped, checked against closed forms the
oracle's cache model gives (every retained key equally weighted; one dominant needle key far
out in the buffer, which also drives the work-group's exact-max fallback).  Also: the bounded
rotary table cache, the step on a stream other than the current one, and a cache restored
from a snapshot of its buffers through unstep_cache_advance.
Inputs from synth or closed-form recipes; expected values from oracle only."""
import math

import numpy as np
import pytest
import torch

from oracle import numerics, rope
from oracle import tables as otables
from oracle.kvcache import KVCacheOracle, retained_frames, slot_of_frame
from tests.gpu_helpers import Mirror, check_attention, dev, host, log

pytestmark = pytest.mark.gpu

u = pytest.importorskip("paper_2609_32518_amd")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

SCALE = 1.0 / math.sqrt(128.0)


def test_single_token_single_key():
    # grid 1x1, one-frame chunks, no window: each query sees exactly its own key, so the output
    # is that key's value row, bit for bit, and the log-sum-exp is the scaled score
    m = Mirror(u, 1, 1, 1, 1, 0, 1)
    for f in range(3):
        q_rot, out, lse, q_want = m.step(f, 1, 0, (40, f), lse=True)
        torch.cuda.synchronize()
        assert np.array_equal(host(q_rot), q_want)
        m.check_cache(f"frame {f}")
        v_row = m.orc.v[0, 0, m.orc.slot(f)]
        assert np.array_equal(host(out).reshape(-1), v_row)
        s = float(np.dot(numerics.bf16_to_f64(q_want.reshape(-1)), numerics.bf16_to_f64(m.orc.k[0, 0, m.orc.slot(f)])))
        assert abs(float(lse.cpu().numpy().reshape(-1)[0]) - s * SCALE) <= 1e-5 * max(1.0, abs(s * SCALE))


def test_zero_window_keeps_sinks_and_chunk():
    m = Mirror(u, 1, 2, 4, 6, 2, 3)
    for c in range(5):
        q_rot, out, _, q_want = m.step(2 * c, 2, 0, (41, c))
        torch.cuda.synchronize()
        m.check_cache(f"chunk {c}")
        assert m.orc.retained(2 * c, 2, 0) == sorted(set(range(min(2, 2 * c))) | {2 * c, 2 * c + 1})
        want, _ = m.expected(q_want, 2 * c, 2, 0)
        check_attention(host(out), want, f"chunk {c}")


def _v_pattern(frames: np.ndarray) -> np.ndarray:
    # value row of every token of frame f: ((3 f + d) mod 8) - 3.5, exact in bf16
    d = np.arange(128)
    return ((3 * frames[:, None] + d[None, :]) % 8).astype(np.float64) - 3.5


def test_maximum_cache_with_wrapped_ring():
    # 64x64 tokens per frame, a ring of 2047 frames: 8,384,512 rows per buffer, the last byte at
    # 2^31 - 1,048,833; the chunk at frame 3047 sees frames 1001-3047 through a wrapped ring
    gh = gw = 64
    T = gh * gw
    R = 2047
    f0 = 3047
    W = R - 1
    rows = R * T
    assert rows <= 8388607 and rows * 256 < 2 ** 31
    k_buf = torch.zeros((1, 1, rows, 128), dtype=torch.bfloat16, device="cuda")
    v_buf = torch.empty((1, 1, rows, 128), dtype=torch.bfloat16, device="cuda")
    cache = u.Cache(1, 1, gh, gw, 0, R, k_cache=k_buf, v_cache=v_buf)
    orc = KVCacheOracle(1, 1, 128, 1, 1, 0, R)       # index model only (one token per frame)
    for start in range(0, f0, R):
        n = min(R, f0 - start)
        cache.advance(start, n)
        orc.append(start, n, np.zeros((1, n, 1, 128), np.uint16), np.zeros((1, n, 1, 128), np.uint16))
    fm, newest = cache.frame_map()
    assert fm == orc.frame_of_slot and newest == f0 - 1
    # value rows of every slot from the frame it holds (device fill from the same recipe)
    pat = torch.from_numpy(_v_pattern(np.array(fm, dtype=np.int64))).to("cuda", torch.bfloat16)   # [R, 128]
    v_buf.view(R, T, 128).copy_(pat[:, None, :].expand(R, T, 128))
    # the chunk: zero keys, pattern values, appended through the library (no queries)
    tables = u.RopeTableCache("cuda")
    cos_t, sin_t = tables.get(f0, 1, gh, gw)
    kz = torch.zeros((1, T, 1, 128), dtype=torch.bfloat16, device="cuda")
    vc = pat.new_tensor(_v_pattern(np.array([f0]))).to(torch.bfloat16).expand(T, 128).reshape(1, T, 1, 128).contiguous()
    cache.unstep_kv_append(f0, 1, None, kz, vc, cos_t, sin_t)
    orc.append(f0, 1, np.zeros((1, 1, 1, 128), np.uint16), np.zeros((1, 1, 1, 128), np.uint16))
    frames = retained_frames(f0, 1, 0, W)
    assert frames == list(range(f0 - W, f0 + 1)) and len(cache.segments(f0, 1, W)) == 2
    n_keys = len(frames) * T
    vals = _v_pattern(np.array(frames))                              # [frames, 128]
    log(f"max cache: {rows} rows per buffer, {n_keys} keys, {len(cache.segments(f0, 1, W))} segments")

    # (a) zero queries: every retained key weighs the same, the output is their mean value row
    q0 = torch.zeros((1, T, 1, 128), dtype=torch.bfloat16, device="cuda")
    out = cache.unstep_window_attn(f0, 1, W, q0)
    torch.cuda.synchronize()
    want = vals.mean(axis=0)
    got = numerics.bf16_to_f64(host(out)).reshape(T, 128)
    assert np.abs(got - want[None, :]).max() <= 2.0 ** -8 * np.abs(want).max() + 1e-3

    # (b) a needle: the last token of the slot nearest the end of the buffer gets key e_0 * kv,
    # every query is e_0 * qv, all other keys are zero; its weight dominates the sum
    slot = R - 1
    f_needle = fm[slot]
    assert f_needle in frames and slot_of_frame(f_needle, 0, R) == slot
    kv, qv = 24.0, 24.0     # score 576: exp(50.9) against 8.4M unit weights; 2^73 > 2^64 forces the exact-max redo
    k_buf[0, 0, (slot + 1) * T - 1, 0] = kv
    v_buf[0, 0, (slot + 1) * T - 1] = torch.full((128,), 3.0, dtype=torch.bfloat16)
    q = torch.zeros((1, T, 1, 128), dtype=torch.bfloat16, device="cuda")
    q[..., 0] = qv
    lse = torch.empty((1, 1, T), dtype=torch.float32, device="cuda")
    out = cache.unstep_window_attn(f0, 1, W, q, lse=lse)
    torch.cuda.synchronize()
    a = kv * qv * SCALE
    others = vals.sum(axis=0) * T - _v_pattern(np.array([f_needle]))[0]
    want = (math.exp(a) * 3.0 + others) / (math.exp(a) + n_keys - 1)
    got = numerics.bf16_to_f64(host(out)).reshape(T, 128)
    log(f"needle: weight {math.exp(a) / (math.exp(a) + n_keys - 1):.6f}, max err {np.abs(got - want).max():.3g}")
    assert np.abs(got - want[None, :]).max() <= 2.0 ** -8 * 3.0 + 1e-3
    want_lse = math.log(math.exp(a) + n_keys - 1)
    assert np.abs(lse.cpu().numpy() - want_lse).max() <= 1e-3


def test_rope_table_cache_is_bounded():
    # least recently used pairs are dropped beyond max_entries and rebuilt identically on demand
    cache = u.RopeTableCache("cuda", max_entries=2)
    a = cache.get(0, 3, 4, 6)
    cache.get(3, 3, 4, 6)
    assert cache.get(0, 3, 4, 6) is a                # a hit refreshes the pair
    cache.get(6, 3, 4, 6)                            # drops (3, 3, ...), the least recently used
    assert len(cache) == 2 and cache.get(0, 3, 4, 6) is a
    c, s = cache.get(3, 3, 4, 6)                     # rebuilt
    torch.cuda.synchronize()
    oc, os_ = otables.rope_tables(3, 3, 4, 6)
    assert np.array_equal(c.cpu().numpy().view(np.uint32), oc.view(np.uint32))
    assert np.array_equal(s.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    assert len(cache) == 2


def test_step_on_a_side_stream_with_wrapper_allocations():
    # the binding allocates q_rot, out and the split-key scratch itself and the work runs on a
    # stream other than the current one (the scratch grows from plain to balanced shapes on the
    # way); results as on the current stream, checked against the oracle
    m = Mirror(u, 1, 2, 30, 52, 0, 12)
    side = torch.cuda.Stream()
    for f0 in range(0, 11):
        m.append(f0, 1, (42, f0))
    torch.cuda.synchronize()
    for n, (f0, W) in enumerate([(11, 0), (11, 11), (11, 11)]):
        q, k, v = m.inputs(1, (43, n))
        cos_t, sin_t = m.tables.get(f0, 1, 30, 52)
        qd, kd, vd = dev(q), dev(k), dev(v)
        side.wait_stream(torch.cuda.current_stream())
        out = m.lib.unstep_step(f0, 1, W, qd, kd, vd, cos_t, sin_t, stream=side)
        side.synchronize()
        c, s = otables.rope_tables(f0, 1, 30, 52)
        m.orc.append(f0, 1, rope.rope_bf16(k, c, s), v)
        m.check_cache(f"side stream call {n}")
        want, _ = m.expected(rope.rope_bf16(q, c, s), f0, 1, W)
        check_attention(host(out), want, f"side stream call {n}")
        del out


def test_snapshot_restore_through_advance():
    # the whole cache state is the K/V buffers plus the frame map: copy the buffers of a cache
    # built by real appends (3 sinks, a ring that has wrapped), record the same frames in a new
    # handle over the copies with unstep_cache_advance, and the restored cache attends and then
    # continues the stream exactly as the original
    m = Mirror(u, 1, 2, 6, 8, 3, 6)
    for f0 in range(0, 15, 3):
        m.append(f0, 3, (44, f0))
    torch.cuda.synchronize()
    k2, v2 = m.lib.k.clone(), m.lib.v.clone()
    r = u.Cache(1, 2, 6, 8, 3, 6, k_cache=k2, v_cache=v2)
    for f0 in range(0, 15, 3):
        r.advance(f0, 3)
    assert r.frame_map() == m.lib.frame_map()
    assert r.segments(12, 3, 3) == m.lib.segments(12, 3, 3)
    for n in range(2):
        q, k, v = m.inputs(3, (45, n))
        cos_t, sin_t = m.tables.get(15 + 3 * n, 3, 6, 8)
        outs = []
        for cache in (m.lib, r):
            outs.append(cache.unstep_step(15 + 3 * n, 3, 3, dev(q), dev(k), dev(v), cos_t, sin_t))
        torch.cuda.synchronize()
        assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16)), n
        assert torch.equal(m.lib.k.view(torch.int16), r.k.view(torch.int16)), n
        assert torch.equal(m.lib.v.view(torch.int16), r.v.view(torch.int16)), n
        c, s = otables.rope_tables(15 + 3 * n, 3, 6, 8)
        m.orc.append(15 + 3 * n, 3, rope.rope_bf16(k, c, s), v)
        want, _ = m.expected(rope.rope_bf16(q, c, s), 15 + 3 * n, 3, 3)
        check_attention(host(outs[1]), want, f"restored cache call {n}")
    m.check_cache("after the restored run")


def _mfma_reference_model(src_bits, groups, wps, mfmas):
    """Each wave's lane-0 checksum of the MFMA rate reference, in float64: lane l of a wave holds
    eight bf16 operand vectors a[s] and eight b[s]; a 32x32x16 MFMA takes A[i][k] from lane
    i + 32 (k // 8), element k % 8, and B[k][j] from lane j + 32 (k // 8); block s of 32 MFMAs
    adds A(a[(j + s) % 8]) B(b[(j // 8 + s) % 8]) into accumulator j % 8, and lane 0 holds
    column 0, rows 0-3, 8-11, 16-19 and 24-27 of each accumulator."""
    vals = (src_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    lanes = vals.reshape(groups, 8, 64, 16, 8)                  # group, wave, lane, vector, element
    rows0 = [r for r in range(32) if (r // 4) % 2 == 0]
    out = np.zeros((groups, 8))
    for g in range(groups):
        for w in range(4 * wps):
            lv = lanes[g, w]

            def mat(vec):                                       # [32, 16] from the 64 lanes' vector `vec`
                return np.concatenate([lv[0:32, vec, :], lv[32:64, vec, :]], axis=1)
            A = [mat(s) for s in range(8)]
            Bt = [mat(8 + s) for s in range(8)]                 # Bt[j][k] = B[k][j]
            acc = [np.zeros((32, 32)) for _ in range(8)]
            for blk in range(mfmas // 32):
                s = blk % 8
                for j in range(32):
                    acc[j % 8] += A[(j + s) % 8] @ Bt[((j // 8) + s) % 8].T
            out[g, w] = sum(acc[i][rows0, 0].sum() for i in range(8))
    return out


@pytest.mark.parametrize("wps,mfmas", [(1, 64), (2, 288)])
def test_mfma_reference_computes_its_products(wps, mfmas):
    # the MFMA rate reference multiplies the operands it was given: per-wave checksums against a
    # float64 model of the MFMA lane layout (288 = 9 blocks: the 8-block loop and a 1-block tail);
    # the waves that do not multiply report zero
    groups = 2
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    src = torch.randn(groups * 512 * 128, generator=g, device="cuda").to(torch.bfloat16)
    got = u.unstep_mfma_reference(src, groups, wps, mfmas)
    torch.cuda.synchronize()
    want = _mfma_reference_model(src.view(torch.int16).cpu().numpy().view(np.uint16), groups, wps, mfmas)
    got = got.cpu().numpy().astype(np.float64)
    assert np.all(got[:, 4 * wps:] == 0)
    scale = np.abs(want[:, :4 * wps]).max() + 1.0
    assert np.abs(got - want).max() <= 1e-5 * scale * mfmas, (got, want)


def test_copy_reference_copies_bits():
    # the append pass's bandwidth reference: three buffers copied bit for bit, a ragged piece count
    n = 3 * 257 * 8 + 8                                   # 16-byte pieces, not a multiple of 256 threads
    src = [torch.randint(-32768, 32767, (n,), dtype=torch.int16, device="cuda") for _ in range(3)]
    dst = [torch.zeros_like(t) for t in src]
    u.unstep_copy3(*src, *dst)
    torch.cuda.synchronize()
    for a, b in zip(src, dst):
        assert torch.equal(a, b)
