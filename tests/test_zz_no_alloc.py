"""The allocation-free attention entry point (unstep_window_attn_noalloc) against
unstep_window_attn with a caller-given workspace, through the C ABI: two balanced (split-key)
calls in a row, the second on a smaller launch that reuses the static scratch the first one
filled, then a plain call.  Outputs and log-sum-exp must be bit-identical to the workspace
entry point's (same kernels, same split), and a sample of rows within the attention tolerance
of the oracle."""
import numpy as np
import pytest
import torch

import synth
from tests.gpu_helpers import LSE_ABS, Mirror, check_attention, host, log, sample_queries

pytestmark = pytest.mark.gpu

u = pytest.importorskip("paper_2609_32518_amd")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)


def _filled(B, H, gh, gw, S, R, C, upto, key):
    m = Mirror(u, B, H, gh, gw, S, R)
    for f0 in range(0, upto, C):
        m.append(f0, C, (key, f0))
    return m


def _both(m, f0, C, W, key):
    """Append the chunk, then attend through both entry points; returns the two (out, lse)
    pairs and the oracle's rotated queries."""
    q, qr_dev, c, s = m.append(f0, C, key, with_q=True)
    from oracle import rope
    q_rot_ref = rope.rope_bf16(q, c, s)
    N = C * m.T
    ws_bytes = m.lib.workspace_bytes(f0, C, W)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    shape = (m.B, N, m.H, 128)
    out_ws = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    out_na = torch.full(shape, 7.0, dtype=torch.bfloat16, device="cuda")
    lse_ws = torch.empty((m.B, m.H, N), dtype=torch.float32, device="cuda")
    lse_na = torch.full((m.B, m.H, N), 7.0, dtype=torch.float32, device="cuda")
    m.lib.unstep_window_attn(f0, C, W, qr_dev, out=out_ws, lse=lse_ws, workspace=ws)
    m.lib.unstep_window_attn_noalloc(f0, C, W, qr_dev, out_na, lse=lse_na)
    torch.cuda.synchronize()
    return ws_bytes, (out_ws, lse_ws), (out_na, lse_na), q_rot_ref


def _check(m, f0, C, W, key, what, split):
    ws_bytes, (o1, l1), (o2, l2), q_rot_ref = _both(m, f0, C, W, key)
    log(f"{what}: scratch {ws_bytes} bytes")
    assert (ws_bytes > 0) == split
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), what
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32)), what
    idx = sample_queries(C * m.T, 96, 31)
    want, want_lse = m.expected(q_rot_ref, f0, C, W, query_idx=idx)
    log(f"  {check_attention(host(o2)[:, idx], want, what)}")
    assert np.max(np.abs(l2.cpu().numpy()[:, :, idx] - want_lse)) <= LSE_ABS
    return ws_bytes


def test_noalloc_equals_workspace_entry_point_on_two_calls_then_a_smaller_one():
    # 1: the unwindowed shape (32760 keys, 256 work-groups: the largest scratch)
    wl = synth.WORKLOADS["unwindowed"]
    a = _filled(wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R, wl.C, wl.f0, 60)
    big = _check(a, wl.f0, wl.C, wl.W, (60, 100), "unwindowed", True)
    # 2: a smaller launch (one-frame chunk over 11 frames: 84 query tiles, 252 work-groups),
    # which reads partials only where it wrote them in the scratch the first call left behind
    b = _filled(1, 12, 30, 52, 0, 12, 1, 11, 61)
    small = _check(b, 11, 1, 11, (61, 100), "one-frame chunk", True)
    assert 0 < small < big
    # 3: a shape that runs one work-group per query tile (no scratch)
    wt = synth.WORKLOADS["tiny"]
    c = _filled(wt.B, wt.H, wt.grid_h, wt.grid_w, wt.S, wt.R, wt.C, wt.f0, 62)
    _check(c, wt.f0, wt.C, wt.W, (62, 100), "tiny", False)
