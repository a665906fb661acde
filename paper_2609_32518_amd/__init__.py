"""Python binding of libunstep.so: the windowed-attention chunk step of a causal video
DiT (UnStep, arXiv 2609.32518) on one AMD MI355X.

Argument marshalling only: every step of the path runs in the library's HIP kernels.
PyTorch provides device memory (tensors) and the stream; the library's C ABI
(include/unstep.h) takes raw pointers.  The binding has the same names as the ABI:
``unstep_rope_tables``, ``unstep_kv_append`` (+ ``_qknorm``), ``unstep_window_attn``, ``unstep_step``
as methods of a ``Cache`` handle (or functions), ``RopeTableCache`` for the per-chunk tables, and
the clip-level calls ``unstep_sampler_calls``, ``unstep_shift_schedule``, ``unstep_renoise``,
``unstep_emit``, ``unstep_svd_truncate`` and ``unstep_linear``.

Importing this package loads libunstep.so and raises if it is missing: there is no
fallback path.  Build it with ``python paper_2609_32518_amd/build.py``.
"""
from __future__ import annotations

import collections
import ctypes
import os
from typing import List, Optional, Tuple

import torch

HEAD_DIM = 128
MAX_SEGMENTS = 4

OK, E_NULL, E_SHAPE, E_RANGE, E_STATE, E_HIP, E_ALIGN, E_HOST = 0, -1, -2, -3, -4, -5, -6, -7
STATUS_NAMES = {OK: "OK", E_NULL: "E_NULL", E_SHAPE: "E_SHAPE", E_RANGE: "E_RANGE", E_STATE: "E_STATE",
                E_HIP: "E_HIP", E_ALIGN: "E_ALIGN", E_HOST: "E_HOST"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libunstep.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2609_32518_amd/build.py` "
                      "(there is no non-HIP fallback)")
lib = ctypes.CDLL(LIB_PATH)

_i32, _i64, _f32, _f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
_vp, _sz = ctypes.c_void_p, ctypes.c_size_t
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pf32 = ctypes.POINTER(ctypes.c_float)

# exported symbol -> (restype, argtypes); mirrors include/unstep.h
SIGNATURES = {
    "unstep_version": (ctypes.c_int, []),
    "unstep_last_error": (ctypes.c_char_p, []),
    "unstep_cache_create": (ctypes.c_int, [ctypes.POINTER(_vp), _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "unstep_cache_destroy": (ctypes.c_int, [_vp]),
    "unstep_cache_frame_map": (ctypes.c_int, [_vp, _pi32, _pi32]),
    "unstep_cache_advance": (ctypes.c_int, [_vp, _i32, _i32]),
    "unstep_window_segments": (ctypes.c_int, [_vp, _i32, _i32, _i32, _pi32, _pi32, _pi32]),
    "unstep_rope_tables_host": (ctypes.c_int, [_i32, _i32, _i32, _i32, _i32, _f64, _pf32, _pf32]),
    "unstep_rope_tables": (ctypes.c_int, [_i32, _i32, _i32, _i32, _i32, _f64, _vp, _vp, _vp]),
    "unstep_kv_append": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp]),
    "unstep_kv_append_qknorm": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _f64,
                                               _vp, _vp]),
    "unstep_attn_workspace_size": (ctypes.c_int, [_vp, _i32, _i32, _i32, ctypes.POINTER(_sz)]),
    "unstep_shift_schedule": (ctypes.c_int, [_i32, _f64, ctypes.POINTER(_f64), ctypes.POINTER(_f64)]),
    "unstep_svd_truncate": (ctypes.c_int, [_vp, _i32, _i32, _i32, _vp, _vp, ctypes.POINTER(_f32), _vp]),
    "unstep_linear": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _vp]),
    "unstep_sampler_calls": (ctypes.c_int, [_i32, _i32, _i32, _f64, _i32, _pi32, _pi32, _pi32, _pi32,
                                            ctypes.POINTER(_f64), ctypes.POINTER(_f64)]),
    "unstep_copy3": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp]),
    "unstep_mfma_reference": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _vp]),
    "unstep_renoise": (ctypes.c_int, [_vp, _vp, _f64, _vp, _i64, _vp]),
    "unstep_emit": (ctypes.c_int, [_vp, _vp, _f64, _vp, _i64, _vp]),
    "unstep_window_attn": (ctypes.c_int, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _f32, _vp, _sz, _vp]),
    "unstep_window_attn_noalloc": (ctypes.c_int, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _f32, _vp]),
    "unstep_step": (ctypes.c_int, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _vp,
                                   _f32, _vp, _sz, _vp]),
}
for _name, (_res, _args) in SIGNATURES.items():
    _fn = getattr(lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args


class UnstepError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


def _check(rc: int) -> None:
    if rc != OK:
        raise UnstepError(rc, lib.unstep_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _used_on(stream: Optional[torch.cuda.Stream], *tensors: Optional[torch.Tensor]) -> None:
    """Tell torch's allocator that work enqueued on `stream` uses these tensors, so that their
    memory is not handed to a new allocation before that work has run.  Needed when `stream`
    is not the current stream, on which the wrappers allocate outputs and scratch."""
    if stream is None or stream == torch.cuda.current_stream():
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def _need(t: Optional[torch.Tensor], name: str, shape: Tuple[int, ...], dtype: torch.dtype, device: torch.device,
          contiguous: bool = True) -> None:
    """Reject a tensor the kernels would misread: wrong dtype, shape, device or layout.  The
    library sees only a pointer, so these checks are the binding's half of the contract of
    include/unstep.h (the library checks sizes, alignment and the cache state)."""
    if t is None:
        raise ValueError(f"{name} is required")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the cache on {device}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def version() -> int:
    return lib.unstep_version()


def unstep_rope_tables_host(start_frame: int, n_frames: int, grid_h: int, grid_w: int,
                            head_dim: int = HEAD_DIM, theta: float = 10000.0):
    """Host (numpy float32) cos/sin tables [N, head_dim/2] built by the library."""
    import numpy as np
    n = n_frames * grid_h * grid_w
    c = np.empty((n, head_dim // 2), dtype=np.float32)
    s = np.empty_like(c)
    _check(lib.unstep_rope_tables_host(start_frame, n_frames, grid_h, grid_w, head_dim, theta,
                                       c.ctypes.data_as(_pf32), s.ctypes.data_as(_pf32)))
    return c, s


def unstep_rope_tables(start_frame: int, n_frames: int, grid_h: int, grid_w: int, head_dim: int = HEAD_DIM,
                       theta: float = 10000.0, device="cuda", stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Device cos/sin tables [N, head_dim/2] float32 (blocking upload)."""
    n = n_frames * grid_h * grid_w
    c = torch.empty((n, head_dim // 2), dtype=torch.float32, device=device)
    s = torch.empty_like(c)
    _check(lib.unstep_rope_tables(start_frame, n_frames, grid_h, grid_w, head_dim, theta, c.data_ptr(),
                                  s.data_ptr(), _stream(stream)))
    _used_on(stream, c, s)
    return c, s


class RopeTableCache:
    """Tables keyed by (start frame, n_frames, grid_h, grid_w, theta), built once and reused
    by every layer and denoising call of that chunk (Appendix A.5).  At most `max_entries`
    pairs are kept, the least recently used dropped first, so an endless stream of chunks
    holds a bounded amount of device memory (a dropped pair is rebuilt if asked for again;
    kernels already queued on the stream keep its memory until they have run)."""

    def __init__(self, device="cuda", max_entries: int = 64):
        if max_entries < 1:
            raise ValueError("max_entries must be >= 1")
        self.device = device
        self.max_entries = max_entries
        self._tables: "collections.OrderedDict[tuple, Tuple[torch.Tensor, torch.Tensor]]" = collections.OrderedDict()

    def __len__(self) -> int:
        return len(self._tables)

    def get(self, start_frame: int, n_frames: int, grid_h: int, grid_w: int, theta: float = 10000.0):
        key = (start_frame, n_frames, grid_h, grid_w, theta)
        if key in self._tables:
            self._tables.move_to_end(key)
        else:
            self._tables[key] = unstep_rope_tables(start_frame, n_frames, grid_h, grid_w, HEAD_DIM, theta,
                                                   self.device)
            while len(self._tables) > self.max_entries:
                self._tables.popitem(last=False)
        return self._tables[key]


class Cache:
    """KV cache of one attention layer: device K/V buffers bf16 [B, H, (S+R)*T, 128] owned by
    this object, host-held positions owned by the library handle."""

    def __init__(self, batch: int, n_heads: int, grid_h: int, grid_w: int, sink_frames: int, ring_frames: int,
                 device="cuda", k_cache: Optional[torch.Tensor] = None, v_cache: Optional[torch.Tensor] = None,
                 head_dim: int = HEAD_DIM):
        self.B, self.H, self.grid_h, self.grid_w = batch, n_heads, grid_h, grid_w
        self.S, self.R = sink_frames, ring_frames
        self.T = grid_h * grid_w
        self.slots = (sink_frames + ring_frames) * self.T
        shape = (batch, n_heads, self.slots, head_dim)
        self.k = k_cache if k_cache is not None else torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self.v = v_cache if v_cache is not None else torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self.device = self.k.device
        _need(self.k, "k_cache", shape, torch.bfloat16, self.device)
        _need(self.v, "v_cache", shape, torch.bfloat16, self.device)
        h = _vp()
        _check(lib.unstep_cache_create(ctypes.byref(h), batch, n_heads, head_dim, grid_h, grid_w, sink_frames,
                                       ring_frames, self.k.data_ptr(), self.v.data_ptr()))
        self.handle = h
        self._ws: Optional[torch.Tensor] = None

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            lib.unstep_cache_destroy(h)
            self.handle = None

    # -- host index state ------------------------------------------------------------
    def frame_map(self) -> Tuple[List[int], int]:
        fm = (ctypes.c_int32 * (self.S + self.R))()
        newest = ctypes.c_int32()
        _check(lib.unstep_cache_frame_map(self.handle, fm, ctypes.byref(newest)))
        return list(fm), newest.value

    def advance(self, start_frame: int, n_frames: int) -> None:
        """Record frames as stored without writing device memory (snapshot restore)."""
        _check(lib.unstep_cache_advance(self.handle, start_frame, n_frames))

    def segments(self, start_frame: int, n_frames: int, window_frames: int) -> List[Tuple[int, int]]:
        r0 = (ctypes.c_int32 * MAX_SEGMENTS)()
        ln = (ctypes.c_int32 * MAX_SEGMENTS)()
        n = ctypes.c_int32()
        _check(lib.unstep_window_segments(self.handle, start_frame, n_frames, window_frames, r0, ln,
                                          ctypes.byref(n)))
        return [(r0[i], ln[i]) for i in range(n.value)]

    def workspace_bytes(self, start_frame: int, n_frames: int, window_frames: int) -> int:
        b = _sz()
        _check(lib.unstep_attn_workspace_size(self.handle, start_frame, n_frames, window_frames, ctypes.byref(b)))
        return b.value

    def workspace(self, start_frame: int, n_frames: int, window_frames: int) -> Optional[torch.Tensor]:
        """Device scratch for split-key attention, grown on demand and kept."""
        need = self.workspace_bytes(start_frame, n_frames, window_frames)
        if need == 0:
            return None
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.k.device)
        return self._ws

    # -- step path --------------------------------------------------------------------
    def _strides(self, x: torch.Tensor, name: str, n_frames: int) -> Tuple[int, int]:
        """(token, head) element strides of a q/k/v input [B, n_frames*T, H, 128]: any token and
        head strides with unit stride on the last axis and the batch stride N * token stride
        (e.g. views into a fused [B, N, 3, H, 128] projection output)."""
        N = n_frames * self.T
        _need(x, name, (self.B, N, self.H, HEAD_DIM), torch.bfloat16, self.device, contiguous=False)
        if x.stride(3) != 1 or (self.B > 1 and x.stride(0) != N * x.stride(1)):
            raise ValueError(f"{name} must have unit stride on the last axis and batch stride N * token stride")
        return x.stride(1), x.stride(2)

    def _qkv_strides(self, q: Optional[torch.Tensor], k: torch.Tensor, v: torch.Tensor,
                     n_frames: int) -> Tuple[int, int]:
        ts, hs = self._strides(k, "k", n_frames)
        if self._strides(v, "v", n_frames) != (ts, hs) or (q is not None and self._strides(q, "q", n_frames) != (ts, hs)):
            raise ValueError("q, k, v must share strides")
        return ts, hs

    def _tables(self, cos_t: torch.Tensor, sin_t: torch.Tensor, n_frames: int) -> None:
        for t, name in ((cos_t, "cos_t"), (sin_t, "sin_t")):
            _need(t, name, (n_frames * self.T, HEAD_DIM // 2), torch.float32, self.device)

    def _chunk_out(self, t: Optional[torch.Tensor], name: str, n_frames: int) -> torch.Tensor:
        """A caller-given bf16 [B, N, H, 128] output checked, or a new one."""
        shape = (self.B, n_frames * self.T, self.H, HEAD_DIM)
        if t is None:
            return torch.empty(shape, dtype=torch.bfloat16, device=self.device)
        _need(t, name, shape, torch.bfloat16, self.device)
        return t

    def _lse(self, lse: Optional[torch.Tensor], n_frames: int) -> None:
        if lse is not None:
            _need(lse, "lse", (self.B, self.H, n_frames * self.T), torch.float32, self.device)

    def _workspace_bytes(self, workspace: Optional[torch.Tensor]) -> int:
        if workspace is None:
            return 0
        if workspace.device != self.device or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous tensor on the cache's device")
        return workspace.numel() * workspace.element_size()

    def unstep_kv_append(self, start_frame: int, n_frames: int, q: Optional[torch.Tensor], k: torch.Tensor,
                         v: torch.Tensor, cos_t: torch.Tensor, sin_t: torch.Tensor,
                         q_rot: Optional[torch.Tensor] = None, stream=None) -> Optional[torch.Tensor]:
        ts, hs = self._qkv_strides(q, k, v, n_frames)
        self._tables(cos_t, sin_t, n_frames)
        if q is not None:
            q_rot = self._chunk_out(q_rot, "q_rot", n_frames)
        _check(lib.unstep_kv_append(self.handle, start_frame, n_frames, _ptr(q), k.data_ptr(), v.data_ptr(), ts, hs,
                                    cos_t.data_ptr(), sin_t.data_ptr(), _ptr(q_rot), _stream(stream)))
        _used_on(stream, q_rot)
        return q_rot

    def unstep_kv_append_qknorm(self, start_frame: int, n_frames: int, q: Optional[torch.Tensor], k: torch.Tensor,
                                v: torch.Tensor, cos_t: torch.Tensor, sin_t: torch.Tensor,
                                q_norm_weight: Optional[torch.Tensor], k_norm_weight: torch.Tensor,
                                norm_eps: float = 1e-6, q_rot: Optional[torch.Tensor] = None,
                                stream=None) -> Optional[torch.Tensor]:
        """unstep_kv_append with the RMS normalisation of q and k over each token's H*128 channels
        (weights: bf16 [H*128])."""
        ts, hs = self._qkv_strides(q, k, v, n_frames)
        self._tables(cos_t, sin_t, n_frames)
        _need(k_norm_weight, "k_norm_weight", (self.H * HEAD_DIM,), torch.bfloat16, self.device)
        if q is not None:
            _need(q_norm_weight, "q_norm_weight", (self.H * HEAD_DIM,), torch.bfloat16, self.device)
            q_rot = self._chunk_out(q_rot, "q_rot", n_frames)
        _check(lib.unstep_kv_append_qknorm(self.handle, start_frame, n_frames, _ptr(q), k.data_ptr(), v.data_ptr(),
                                           ts, hs, cos_t.data_ptr(), sin_t.data_ptr(), _ptr(q_norm_weight),
                                           k_norm_weight.data_ptr(), norm_eps, _ptr(q_rot), _stream(stream)))
        _used_on(stream, q_rot)
        return q_rot

    def unstep_window_attn(self, start_frame: int, n_frames: int, window_frames: int, q_rot: torch.Tensor,
                           out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                           softmax_scale: float = 0.0, workspace: Optional[torch.Tensor] = None,
                           use_split: bool = True, stream=None) -> torch.Tensor:
        _need(q_rot, "q_rot", (self.B, n_frames * self.T, self.H, HEAD_DIM), torch.bfloat16, self.device)
        out = self._chunk_out(out, "out", n_frames)
        self._lse(lse, n_frames)
        if workspace is None and use_split:
            workspace = self.workspace(start_frame, n_frames, window_frames)
        ws_bytes = self._workspace_bytes(workspace)
        _check(lib.unstep_window_attn(self.handle, start_frame, n_frames, window_frames, q_rot.data_ptr(),
                                      out.data_ptr(), _ptr(lse), softmax_scale, _ptr(workspace), ws_bytes,
                                      _stream(stream)))
        _used_on(stream, out, workspace)
        return out

    def unstep_window_attn_noalloc(self, start_frame: int, n_frames: int, window_frames: int, q_rot: torch.Tensor,
                                   out: torch.Tensor, lse: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                                   stream=None) -> torch.Tensor:
        """unstep_window_attn with the split-key scratch in the library's static device array (no
        workspace, no allocation in the library; the caller passes the output).  Calls that may
        overlap on one device race on that array."""
        _need(q_rot, "q_rot", (self.B, n_frames * self.T, self.H, HEAD_DIM), torch.bfloat16, self.device)
        _need(out, "out", (self.B, n_frames * self.T, self.H, HEAD_DIM), torch.bfloat16, self.device)
        self._lse(lse, n_frames)
        _check(lib.unstep_window_attn_noalloc(self.handle, start_frame, n_frames, window_frames, q_rot.data_ptr(),
                                              out.data_ptr(), _ptr(lse), softmax_scale, _stream(stream)))
        return out

    def unstep_step(self, start_frame: int, n_frames: int, window_frames: int, q: torch.Tensor, k: torch.Tensor,
                    v: torch.Tensor, cos_t: torch.Tensor, sin_t: torch.Tensor, q_rot: Optional[torch.Tensor] = None,
                    out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                    softmax_scale: float = 0.0, workspace: Optional[torch.Tensor] = None, use_split: bool = True,
                    stream=None) -> torch.Tensor:
        if q is None:
            raise ValueError("unstep_step needs q")
        ts, hs = self._qkv_strides(q, k, v, n_frames)
        self._tables(cos_t, sin_t, n_frames)
        q_rot = self._chunk_out(q_rot, "q_rot", n_frames)
        out = self._chunk_out(out, "out", n_frames)
        self._lse(lse, n_frames)
        if workspace is None and use_split:
            workspace = self._step_workspace(start_frame, n_frames, window_frames)
        ws_bytes = self._workspace_bytes(workspace)
        _check(lib.unstep_step(self.handle, start_frame, n_frames, window_frames, q.data_ptr(), k.data_ptr(),
                               v.data_ptr(), ts, hs, cos_t.data_ptr(), sin_t.data_ptr(), q_rot.data_ptr(),
                               out.data_ptr(), _ptr(lse), softmax_scale, _ptr(workspace), ws_bytes,
                               _stream(stream)))
        _used_on(stream, q_rot, out, workspace)
        return out

    def _step_workspace(self, start_frame: int, n_frames: int, window_frames: int) -> Optional[torch.Tensor]:
        return self.workspace(start_frame, n_frames, window_frames)


# -- clean-cache updates (Section 3.4) ---------------------------------------------------------
def unstep_shift_schedule(n_steps: int = 4, shift: float = 5.0):
    """(sigma, t) float64 numpy arrays of the shifted n-step schedule, built by the library."""
    import numpy as np
    sigma = np.zeros(n_steps, np.float64)
    t = np.zeros(n_steps, np.float64)
    _check(lib.unstep_shift_schedule(n_steps, shift, sigma.ctypes.data_as(ctypes.POINTER(_f64)),
                                     t.ctypes.data_as(ctypes.POINTER(_f64))))
    return sigma, t


# -- V/O truncated SVD and the projection after attention (Section 3.5, Appendix A.4) -------------
def unstep_svd_truncate(w: torch.Tensor, rank: int, bf16: bool = True, stream=None):
    """Init-time rank-r reconstruction of a float32 [rows, cols] device weight.  Returns
    (w_r float32, w_r bf16 or None, singular values as a float32 numpy array)."""
    import numpy as np
    if w.dtype != torch.float32 or w.dim() != 2 or not w.is_contiguous():
        raise ValueError("w must be a contiguous float32 matrix")
    rows, cols = w.shape
    w_r = torch.empty_like(w)
    w_b = torch.empty((rows, cols), dtype=torch.bfloat16, device=w.device) if bf16 else None
    sig = np.zeros(min(rows, cols), np.float32)
    _check(lib.unstep_svd_truncate(w.data_ptr(), rows, cols, rank, w_r.data_ptr(), _ptr(w_b),
                                   sig.ctypes.data_as(ctypes.POINTER(_f32)), _stream(stream)))
    return w_r, w_b, sig


def unstep_linear(x: torch.Tensor, w: torch.Tensor, bias: Optional[torch.Tensor] = None,
                  out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """y = x W^T + b for bf16 x [..., K], W [N, K], b [N]."""
    for t in (x, w) + ((bias,) if bias is not None else ()):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError("x, w, bias must be contiguous bf16 tensors")
    N, K = w.shape
    if x.shape[-1] != K or (bias is not None and bias.shape != (N,)):
        raise ValueError("shapes: x [..., K], w [N, K], bias [N]")
    M = x.numel() // K
    for t in (w,) + ((bias,) if bias is not None else ()):
        if t.device != x.device:
            raise ValueError("x, w, bias must be on one device")
    if out is None:
        out = torch.empty(x.shape[:-1] + (N,), dtype=torch.bfloat16, device=x.device)
    else:
        _need(out, "out", tuple(x.shape[:-1]) + (N,), torch.bfloat16, x.device)
    _check(lib.unstep_linear(x.data_ptr(), w.data_ptr(), _ptr(bias), out.data_ptr(), M, N, K, _stream(stream)))
    _used_on(stream, out)
    return out


SAMPLERS = {"self_forcing": 0, "unstep": 1, "unstep_one_step": 2}
SCHEDULE_CLEAN = -1


def unstep_sampler_calls(variant: str, n_chunks: int, chunk_frames: int = 3, clean_sigma: Optional[float] = None):
    """The clip's DiT calls from the library: dict of numpy arrays chunk, start_frame,
    schedule_index (SCHEDULE_CLEAN for the clean-cache call), sigma, t."""
    import numpy as np
    if variant not in SAMPLERS:
        raise ValueError(f"unknown sampler {variant!r}")
    cs = -1.0 if clean_sigma is None else float(clean_sigma)
    n = _i32(0)
    rc = lib.unstep_sampler_calls(SAMPLERS[variant], n_chunks, chunk_frames, cs, 0, ctypes.byref(n), None, None, None,
                                  None, None)
    if rc not in (0, -3) or (rc == -3 and n.value == 0):
        _check(rc)
    cap = n.value
    out = dict(chunk=np.zeros(cap, np.int32), start_frame=np.zeros(cap, np.int32),
               schedule_index=np.zeros(cap, np.int32), sigma=np.zeros(cap, np.float64), t=np.zeros(cap, np.float64))
    p32 = lambda a: a.ctypes.data_as(_pi32)
    p64 = lambda a: a.ctypes.data_as(ctypes.POINTER(_f64))
    _check(lib.unstep_sampler_calls(SAMPLERS[variant], n_chunks, chunk_frames, cs, cap, ctypes.byref(n),
                                    p32(out["chunk"]), p32(out["start_frame"]), p32(out["schedule_index"]),
                                    p64(out["sigma"]), p64(out["t"])))
    return out


def _latent(x: torch.Tensor) -> None:
    if x.dtype != torch.bfloat16 or not x.is_contiguous():
        raise ValueError("latents must be contiguous bf16 tensors")


def unstep_renoise(x: torch.Tensor, eps: torch.Tensor, sigma: float, out: Optional[torch.Tensor] = None,
                   stream=None) -> torch.Tensor:
    """Equation 1: (1 - sigma) x + sigma eps."""
    for t in (x, eps):
        _latent(t)
    if eps.shape != x.shape:
        raise ValueError("x and eps must have the same shape")
    if eps.device != x.device:
        raise ValueError("x and eps must be on one device")
    out = torch.empty_like(x) if out is None else out
    _need(out, "out", tuple(x.shape), torch.bfloat16, x.device)
    _check(lib.unstep_renoise(x.data_ptr(), eps.data_ptr(), sigma, out.data_ptr(), x.numel(), _stream(stream)))
    _used_on(stream, out)
    return out


def unstep_emit(x_tilde: torch.Tensor, v: torch.Tensor, sigma: float, out: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """Equation 3: x_tilde - sigma v."""
    for t in (x_tilde, v):
        _latent(t)
    if v.shape != x_tilde.shape:
        raise ValueError("x_tilde and v must have the same shape")
    if v.device != x_tilde.device:
        raise ValueError("x_tilde and v must be on one device")
    out = torch.empty_like(x_tilde) if out is None else out
    _need(out, "out", tuple(x_tilde.shape), torch.bfloat16, x_tilde.device)
    _check(lib.unstep_emit(x_tilde.data_ptr(), v.data_ptr(), sigma, out.data_ptr(), x_tilde.numel(), _stream(stream)))
    _used_on(stream, out)
    return out


def unstep_copy3(a: torch.Tensor, b: torch.Tensor, c: torch.Tensor, x: torch.Tensor, y: torch.Tensor,
                 z: torch.Tensor, stream=None) -> None:
    """x = a, y = b, z = c in one launch with the append pass's access pattern (a bandwidth
    reference for that pass, not part of the method)."""
    n = a.numel() * a.element_size()
    for t in (a, b, c, x, y, z):
        if not t.is_contiguous() or t.numel() * t.element_size() != n or t.device != a.device:
            raise ValueError("six contiguous buffers of one size on one device")
    _check(lib.unstep_copy3(a.data_ptr(), b.data_ptr(), c.data_ptr(), x.data_ptr(), y.data_ptr(), z.data_ptr(), n,
                            _stream(stream)))


def unstep_mfma_reference(src: torch.Tensor, groups: int, waves_per_simd: int, mfmas: int,
                          out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The MFMA rate reference (not part of the method): `groups` work-groups of 8 waves,
    `waves_per_simd` multiplying waves per SIMD, each running `mfmas` bf16 MFMAs on operands read
    once from src (bf16, contiguous, groups * 512 * 128 values).  Returns the per-wave checksums,
    fp32 [groups, 8]."""
    _need(src, "src", (groups * 512 * 128,), torch.bfloat16, src.device)
    if out is None:
        out = torch.empty((groups, 8), dtype=torch.float32, device=src.device)
    _need(out, "out", (groups, 8), torch.float32, src.device)
    _check(lib.unstep_mfma_reference(src.data_ptr(), out.data_ptr(), groups, waves_per_simd, mfmas, _stream(stream)))
    _used_on(stream, src, out)
    return out
