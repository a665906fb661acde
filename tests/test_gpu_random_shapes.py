"""GPU parity over seeded random small shapes (tests/gpu_helpers.random_shape_cases): batch,
heads, grid, sinks, ring, chunk and window drawn at random, each case a stream of chunk steps
through unstep_step (repeats of the newest chunk included) on the balanced or the plain
schedule; every third case again through the RMS-norm append.  After every call q_rot, both
caches and the frame map are bit-exact and the attention output (and the log-sum-exp where
requested) within the stated tolerance of the oracle.  Inputs from synth only; expected values from oracle only."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_helpers import LSE_ABS, Mirror, check_attention, host, log, random_medium_cases, random_shape_cases

pytestmark = pytest.mark.gpu

u = pytest.importorskip("paper_2609_32518_amd")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

CASES = random_shape_cases()
MEDIUM = random_medium_cases()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_random_shape_stream(case):
    _stream(CASES[case], case)


@pytest.mark.parametrize("case", range(len(MEDIUM)))
def test_random_medium_shape_stream(case):
    _stream(MEDIUM[case], 100 + case)


def _stream(cs, case):
    C, W = cs["C"], cs["W"]
    log(f"random shape {case}: " + " ".join(f"{k}={v}" for k, v in cs.items() if k != "calls"))
    m = Mirror(u, cs["B"], cs["H"], cs["gh"], cs["gw"], cs["S"], cs["R"])
    for n, (f0, use_split, with_lse) in enumerate(cs["calls"]):
        what = f"case {case} call {n} (f0 {f0}, split {use_split})"
        q_rot, out, lse, q_ref = m.step(f0, C, W, (5000 + case, n), use_split=use_split, lse=with_lse)
        torch.cuda.synchronize()
        assert np.array_equal(host(q_rot), q_ref), f"{what}: q_rot"
        m.check_cache(what)
        want, want_lse = m.expected(q_ref, f0, C, W)
        check_attention(host(out), want, what)
        if with_lse:
            assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS, f"{what}: lse"


@pytest.mark.parametrize("case", range(0, len(CASES), 3))
def test_random_shape_stream_qknorm(case):
    # every third case again through the fused RMS-norm + RoPE append (unstep_kv_append_qknorm),
    # fused [B, N, 3, H, D] strides on odd calls, then windowed attention on the normalised cache
    cs = CASES[case]
    C, W, H = cs["C"], cs["W"], cs["H"]
    log(f"random shape qknorm {case}: " + " ".join(f"{k}={v}" for k, v in cs.items() if k != "calls"))
    m = Mirror(u, cs["B"], H, cs["gh"], cs["gw"], cs["S"], cs["R"])
    gen = synth.generator(6000, case)
    wq = synth.bf16_bits_from_f32(1.0 + 0.1 * gen.standard_normal(H * 128).astype(np.float32))
    wk = synth.bf16_bits_from_f32(1.0 + 0.1 * gen.standard_normal(H * 128).astype(np.float32))
    for n, (f0, use_split, with_lse) in enumerate(cs["calls"]):
        what = f"qknorm case {case} call {n} (f0 {f0}, split {use_split})"
        qr, q_ref = m.append_qknorm(f0, C, (6000 + case, n), wq, wk,
                                    q_layout="fused_qkv" if n % 2 else "contiguous")
        lse = torch.empty((cs["B"], H, C * m.T), dtype=torch.float32, device="cuda") if with_lse else None
        out = m.lib.unstep_window_attn(f0, C, W, qr, lse=lse, use_split=use_split)
        torch.cuda.synchronize()
        assert np.array_equal(host(qr), q_ref), f"{what}: q_rot"
        m.check_cache(what)
        want, want_lse = m.expected(q_ref, f0, C, W)
        check_attention(host(out), want, what)
        if with_lse:
            assert np.max(np.abs(lse.cpu().numpy() - want_lse)) <= LSE_ABS, f"{what}: lse"
