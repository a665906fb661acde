"""Benchmark of the windowed-attention chunk step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--sub-steps K2] [--sets 6] [--no-cpu-baseline]

A step is one whole pass of the hot path over one chunk: the fused RoPE + KV append
and the windowed attention (unstep_step).  The default workload is the full-frame
chunk: 12 heads of width 128, a 30x52 token grid, a 3-frame chunk (4680 queries) at
latent frame 9 over 9 prior frames (18720 retained keys).  Other workloads:
unwindowed (32760 keys), paper_default (3 sinks + 6 recent frames, 14040 keys),
short_refine (one step = 30 layers x 2 calls over 9360 keys), rolling (one step =
60 one-frame chunks through a 12-frame ring from empty) and tiny (2 heads, 4x6 grid).
Without --workload the run times the full-frame chunk as the headline (`value`,
`roofline`, `cpu_baseline`) and then every other workload, each as a record under
`workloads` (attention and append per call with their roofline fractions, the step; the
short-window refine also its 60-call attention total, the rolling stream the mean, min and
max of its per-chunk attention times); --workload NAME times only that one.

Inputs are synthetic, seeded N(0,1) bf16, resident in HBM before timing.  Several
buffer sets (cache + inputs + outputs) are rotated so that consecutive steps do not
find their data in the 256 MB Infinity Cache.  W warm-up steps, then K timed steps
between device synchronisations (`value`, `ms_per_step`).  Then K more steps in which
each call's attention (and, in the balanced schedule, its merge) sits between two HIP
events recorded on its stream, the call enqueued as its two entry points (append, then
attention: the kernels of unstep_step, in its order); the median over the steps of
each call's event interval is the attention duration of `attn` and `roofline`.  Then
each kernel of the step runs on its own for the same calls,
back to back between two events after an untimed pass (which loads the kernels):
the append (`rope_roofline`) and its bandwidth reference, a plain three-buffer copy of
the append pass's inputs (unstep_copy3, `append_copy_baseline`), enqueued behind a
device-side spin so that the events bracket GPU time only with no host enqueue gap,
and the attention alone (`attn.us_per_call_back_to_back`).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "windowed-attn TFLOP/s + µs per chunk-step (12×128 heads, 4680 q); RoPE GB/s"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E, published


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    # the GPU settles its clock under sustained MFMA load within ~20 ms: warm up past that
    p.add_argument("--warmup", type=int, default=40)
    p.add_argument("--workload", default=None,
                   help="time only this workload (default: the full-frame chunk as the headline, plus a "
                        "record per other workload)")
    p.add_argument("--sub-steps", type=int, default=10, help="timed steps of each other workload's record")
    p.add_argument("--sub-warmup", type=int, default=10)
    p.add_argument("--sets", type=int, default=6)
    p.add_argument("--no-split", action="store_true",
                   help="attention without a workspace: one work-group per query tile over its whole key "
                        "range, whatever the plan would pick")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--qknorm", action="store_true",
                   help="append with the fused RMS normalisation of q and k (unstep_kv_append_qknorm), "
                        "then attention, instead of unstep_step")
    p.add_argument("--cpu-queries", type=int, default=0,
                   help="oracle sample: queries x all heads (0 = every query of the chunk, ~4 s on 16 cores)")
    p.add_argument("--flow-update", action="store_true",
                   help="only time the clean-cache renoise + emit updates on one chunk's latent "
                        "(1 x 16 x 3 x 60 x 104 bf16) and print their own JSON line")
    p.add_argument("--oproj", action="store_true",
                   help="time the projection after attention (y = x W^T + b, 4680 x 1536 x 1536 bf16) and "
                        "the init-time V/O truncated SVD of one 1536 x 1536 weight; print their own JSON line")
    p.add_argument("--clip", default=None, choices=["unstep", "unstep_one_step", "self_forcing"],
                   help="time whole clips instead: the sampler's DiT calls (renoise, one chunk step per "
                        "attention layer, emit) and print their own JSON line (--clips, --warmup-clips)")
    p.add_argument("--clip-chunks", type=int, default=7,
                   help="chunks per clip (7 = the 21 latent frames of an 81-frame, 5 s clip; 41 for 30 s)")
    p.add_argument("--clips", type=int, default=3, help="timed clips (with --clip)")
    p.add_argument("--warmup-clips", type=int, default=1)
    p.add_argument("--layers", type=int, default=30)
    p.add_argument("--eight-frame-layers", default="odd",
                   help="layers keeping eight frames (two sinks) instead of nine: 'none', 'all', 'odd', "
                        "or comma-separated layer indices (the paper does not list them)")
    p.add_argument("--summarize-clip-profile", metavar="DIR", default=None,
                   help="read the kernel trace of a profiled --clip run under DIR and write "
                        "profiles/kernels_clip_<variant>.md (pass the same --clip arguments)")
    p.add_argument("--summarize-profile", metavar="DIR", default=None,
                   help="read the rocprofv3 CSV output of the profiling commands under DIR (see "
                        "profile_commands()), write profiles/<kernel>_<workload>.md and "
                        "profiles/traffic.json, and exit")
    p.add_argument("--summarize-trace", metavar="DIR", default=None,
                   help="write profiles/kernels_<--trace-name>.md from the rocprofv3 --kernel-trace --stats "
                        "output in DIR (any bench mode; --trace-command is the command that made it)")
    p.add_argument("--trace-name", default=None)
    p.add_argument("--trace-command", default=None)
    p.add_argument("--mfma-reference", action="store_true",
                   help="time the MFMA rate reference (bf16 MFMAs alone, random operands) in the launch shapes "
                        "of the full-frame chunk's attention and of its output projection")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                   help="only run a plain device-to-device copy of MB megabytes (x5), for scaling HBM "
                        "byte counters read by a profiler")
    return p.parse_args()


def timed_passes(torch, enqueue, passes, spin=True, batch=128):
    """Run enqueue() `passes` times between HIP events on the current stream after one untimed
    pass (which also loads the kernels and sizes the wait); returns ms per pass.  spin: for
    launches short against the binding's host time, enqueue the passes in batches of `batch`,
    each behind a device-side spin long enough for the host to enqueue the whole batch first (a
    batch fits the hardware queue), so that the events bracket GPU time only, with no host
    enqueue gap between launches."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    enqueue()
    t_host = time.perf_counter() - t0
    torch.cuda.synchronize()
    batch = batch if spin else passes
    total_ms, done = 0.0, 0
    while done < passes:
        n = min(batch, passes - done)
        if spin:
            wait_s = min(1.0, 2.0 * t_host * n + 2e-3)
            torch.cuda._sleep(int(wait_s * 2.5e9))   # spin counted in shader cycles (<= 2.4 GHz)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            enqueue()
        e1.record()
        torch.cuda.synchronize()
        total_ms += e0.elapsed_time(e1)
        done += n
    return total_ms / passes


def attn_flops(H, Nq, Nk, D=128):
    return 4.0 * H * Nq * Nk * D


def rope_bytes(H, Nq, D=128):
    # read q, k, v + write q_rot, K row, V row (bf16) + cos, sin (fp32, D/2 each) per token
    return Nq * (12 * H * D + 4 * D)


class Plan:
    """The step's work for one workload: a list of (cache set, start frame, frames, window)."""

    def __init__(self, u, torch, wl, n_sets, qknorm=False, no_split=False):
        self.u, self.torch, self.wl = u, torch, wl
        dev = "cuda"
        g = torch.Generator(device=dev)
        N = wl.n_query

        def randn(shape, seed):
            g.manual_seed(seed)
            return torch.randn(shape, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)

        self.qknorm = qknorm
        self.no_split = no_split
        if qknorm:
            # learned-norm-like weights around 1
            g.manual_seed(7)
            self.wq = (1.0 + 0.1 * torch.randn(wl.H * 128, generator=g, device=dev)).to(torch.bfloat16)
            self.wk = (1.0 + 0.1 * torch.randn(wl.H * 128, generator=g, device=dev)).to(torch.bfloat16)

        self.tables = u.RopeTableCache(dev)
        self.sets = []
        if wl.name == "short_refine":
            n_caches = wl.layers                      # one cache per layer; the layers rotate HBM
        elif wl.name == "rolling":
            n_caches = n_sets
        else:
            n_caches = n_sets
        for si in range(n_caches):
            cache = u.Cache(wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R, device=dev)
            shape = (wl.B, N, wl.H, 128)
            s = dict(cache=cache, q=randn(shape, 10 * si + 1), k=randn(shape, 10 * si + 2),
                     v=randn(shape, 10 * si + 3), q_rot=torch.empty(shape, dtype=torch.bfloat16, device=dev),
                     out=torch.empty(shape, dtype=torch.bfloat16, device=dev))
            if wl.name != "rolling":
                self._prefill(cache, randn, 1000 * (si + 1))
            self.sets.append(s)
        # per step: list of (set index, start frame, frames, window)
        if wl.name == "short_refine":
            self.calls = [(layer, wl.f0, wl.C, wl.W) for layer in range(wl.layers) for _ in range(wl.passes)]
        elif wl.name == "rolling":
            self.calls = [(None, c, 1, wl.W) for c in range(wl.chunks)]
        else:
            self.calls = [(None, wl.f0, wl.C, wl.W)]
        for (_, f0, C, W) in self.calls:
            self.tables.get(f0, C, wl.grid_h, wl.grid_w)
        self.ws = {}
        for si, s in enumerate(self.sets if not no_split else []):
            for (_, f0, C, W) in self.calls:
                need = s["cache"].workspace_bytes(f0, C, W)
                if need and need > self.ws.get(si, torch.empty(0)).numel():
                    self.ws[si] = torch.empty(need, dtype=torch.uint8, device=dev)
        self.step_idx = 0

    def attn_launch_shape(self, f0, C, W):
        """(work-groups, MFMAs per multiplying wave) of the attention launch of a call: one
        work-group per 256-query tile walking all its key tiles (one M phase more than tiles),
        or the balanced split's work-groups (from the workspace the call needs), each walking
        about its share of the (query tile, key tile) units in up to two segments."""
        wl = self.wl
        qtiles = wl.B * wl.H * -(-C * wl.T // 256)
        tk = -(-self.keys(f0, C, W) // 64)
        need = 0 if self.no_split else self.sets[0]["cache"].workspace_bytes(f0, C, W)
        if need == 0:
            return qtiles, 32 * (tk + 1)
        groups = need // (2 * 256 * 130 * 4)
        return groups, 32 * (-(-qtiles * tk // groups) + 2)

    def _prefill(self, cache, randn, seed):
        wl = self.wl
        for f0 in range(0, wl.f0, wl.C):
            shape = (wl.B, wl.C * wl.T, wl.H, 128)
            cos_t, sin_t = self.tables.get(f0, wl.C, wl.grid_h, wl.grid_w)
            cache.unstep_kv_append(f0, wl.C, None, randn(shape, seed + f0), randn(shape, seed + f0 + 500), cos_t,
                                   sin_t)

    def keys(self, f0, C, W):
        wl = self.wl
        lo = max(0, f0 - W)
        return (min(wl.S, lo) + f0 + C - lo) * wl.T

    def per_step(self):
        wl = self.wl
        fl = sum(attn_flops(wl.H, C * wl.T, self.keys(f0, C, W)) * wl.B for (_, f0, C, W) in self.calls)
        by = sum(self.append_bytes(C) for (_, f0, C, W) in self.calls)
        return fl, by

    def append_bytes(self, C):
        wl = self.wl
        # the normalising pass also reads the two weight vectors (bf16 [H*128]) once
        return rope_bytes(wl.H, C * wl.T) * wl.B + (4 * wl.H * 128 if self.qknorm else 0)

    def _append(self, s, f0, C, q, k, v, cos_t, sin_t, q_rot):
        if self.qknorm:
            s["cache"].unstep_kv_append_qknorm(f0, C, q, k, v, cos_t, sin_t, self.wq, self.wk, q_rot=q_rot)
        else:
            s["cache"].unstep_kv_append(f0, C, q, k, v, cos_t, sin_t, q_rot=q_rot)

    def _set_for(self, call_set):
        if call_set is not None:
            return call_set
        return self.step_idx % len(self.sets)

    def behind_wait(self, enqueue, steps, spin=True, launches_per_pass=1):
        """timed_passes() on this plan's torch; spin only for kernels short against the host
        time: kernels much longer than it (attention) run without the spin, since a spin leaves
        the power-limited chip in a different clock state than the step loop does.  Returns ms
        per pass."""
        return timed_passes(self.torch, enqueue, steps, spin, max(1, 128 // max(1, launches_per_pass)))

    def time_kernels(self, steps):
        """Average per-step time (ms) of the appends and of the attention calls, each launched
        for `steps` steps back to back (behind_wait)."""
        out = []
        for which in ("append", "attn"):
            self.step_idx = 0
            out.append(self.behind_wait(lambda: self.step(only=which), steps, spin=which == "append",
                                        launches_per_pass=len(self.calls)))
        return out

    def time_rolling(self, steps):
        """The rolling stream's kernels, each kind back to back: the appends of the 60 chunks on a
        fresh ring (one event pair around each step's appends, behind the spin: they are short),
        then the attention calls with an event pair around each (its key range grows over the
        stream), the host index advanced between them without device work
        (unstep_cache_advance) so that each call attends the key range its chunk has; the
        timing does not depend on what the ring holds.  Returns (append ms per step, attention
        ms per call over all timed steps in chunk order)."""
        torch, wl = self.torch, self.wl
        att = []

        def one_step(which):
            s = self.sets[self.step_idx % len(self.sets)]
            cache = self.u.Cache(wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R, k_cache=s["cache"].k,
                                 v_cache=s["cache"].v)
            for (_, f0, C, W) in self.calls:
                N = C * wl.T
                if which == "append":
                    cos_t, sin_t = self.tables.get(f0, C, wl.grid_h, wl.grid_w)
                    self._append(dict(s, cache=cache), f0, C, s["q"][:, :N], s["k"][:, :N], s["v"][:, :N],
                                 cos_t, sin_t, s["q_rot"][:, :N])
                else:
                    cache.advance(f0, C)
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record()
                    cache.unstep_window_attn(f0, C, W, s["q_rot"][:, :N], out=s["out"][:, :N],
                                             workspace=self.ws.get(self.step_idx % len(self.sets)),
                                             use_split=not self.no_split)
                    b.record()
                    att.append((a, b))
            self.step_idx += 1

        self.step_idx = 0
        app_ms = self.behind_wait(lambda: one_step("append"), steps, spin=True, launches_per_pass=len(self.calls))
        self.step_idx = 0
        self.behind_wait(lambda: one_step("attn"), steps, spin=False)
        return app_ms, [a.elapsed_time(b) for (a, b) in att[len(self.calls):]]    # the untimed pass dropped

    def time_copy_baseline(self, steps):
        """Average per-step time (ms) of a plain three-buffer copy of each call's q, k, v (the
        append pass's inputs) into three other buffers, one launch per call with the pass's
        access pattern (unstep_copy3), over the same rotating buffer sets (behind_wait)."""
        torch, wl = self.torch, self.wl
        if not hasattr(self, "copy_dst"):
            self.copy_dst = [tuple(torch.empty_like(s["q"]) for _ in range(3)) for s in self.sets]

        def one_step():
            for (cs, f0, C, W) in self.calls:
                si = self._set_for(cs)
                s, d = self.sets[si], self.copy_dst[si]
                N = C * wl.T
                self.u.unstep_copy3(s["q"][:, :N], s["k"][:, :N], s["v"][:, :N], d[0][:, :N], d[1][:, :N],
                                    d[2][:, :N])
            self.step_idx += 1

        self.step_idx = 0
        return self.behind_wait(one_step, steps, spin=True, launches_per_pass=len(self.calls))

    def step(self, only=None, attn_events=None):
        """Enqueue one step (only="append" / "attn": just that kernel of each call).  attn_events:
        a list to which the step appends one (start, end) HIP event pair per call, recorded on the
        current stream around that call's attention (and, in the balanced schedule, its merge);
        the call is then enqueued as its two entry points, the append and the attention, which
        launch the same kernels in the same order as unstep_step."""
        wl = self.wl
        if wl.name == "rolling":
            si = self.step_idx % len(self.sets)
            s = self.sets[si]
            s["cache"] = self.u.Cache(wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R, k_cache=s["cache"].k,
                                      v_cache=s["cache"].v)
        for (cs, f0, C, W) in self.calls:
            si = self._set_for(cs)
            s = self.sets[si]
            N = C * wl.T
            cos_t, sin_t = self.tables.get(f0, C, wl.grid_h, wl.grid_w)
            q, k, v = s["q"][:, :N], s["k"][:, :N], s["v"][:, :N]
            q_rot, out = s["q_rot"][:, :N], s["out"][:, :N]
            ws = self.ws.get(si)
            if only == "append":
                self._append(s, f0, C, q, k, v, cos_t, sin_t, q_rot)
            elif only == "attn":
                s["cache"].unstep_window_attn(f0, C, W, q_rot, out=out, workspace=ws, use_split=not self.no_split)
            elif attn_events is not None:
                self._append(s, f0, C, q, k, v, cos_t, sin_t, q_rot)
                e0, e1 = self.torch.cuda.Event(enable_timing=True), self.torch.cuda.Event(enable_timing=True)
                e0.record()
                s["cache"].unstep_window_attn(f0, C, W, q_rot, out=out, workspace=ws, use_split=not self.no_split)
                e1.record()
                attn_events.append((e0, e1))
            elif not self.qknorm:
                s["cache"].unstep_step(f0, C, W, q, k, v, cos_t, sin_t, q_rot=q_rot, out=out, workspace=ws,
                                       use_split=not self.no_split)
            else:
                self._append(s, f0, C, q, k, v, cos_t, sin_t, q_rot)
                s["cache"].unstep_window_attn(f0, C, W, q_rot, out=out, workspace=ws, use_split=not self.no_split)
        self.step_idx += 1


def cpu_baseline(wl, n_queries):
    """The oracle, untuned, on a bounded sample of the workload: RoPE of one chunk's q and k,
    then exact attention of n_queries queries (all heads) over the retained keys."""
    import numpy as np

    import synth
    from oracle import attention, rope, tables
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    N = wl.n_query
    shape = (wl.B, N, wl.H, 128)
    q = synth.normal_bf16(shape, (90, synth.Q))
    k = synth.normal_bf16(shape, (90, synth.K))
    nk = (min(wl.S, max(0, wl.f0 - wl.W)) + wl.f0 + wl.C - max(0, wl.f0 - wl.W)) * wl.T
    kc = synth.normal_bf16((wl.B, wl.H, nk, 128), (90, synth.CACHE_K))
    vc = synth.normal_bf16((wl.B, wl.H, nk, 128), (90, synth.CACHE_V))
    nq = min(n_queries, N) if n_queries > 0 else N
    # the sample is repeated until at least 10 s of host time have passed (at most 8 times)
    reps, t0 = 0, time.perf_counter()
    while True:
        c, s = tables.rope_tables(wl.f0, wl.C, wl.grid_h, wl.grid_w)
        qr = rope.rope_bf16(q, c, s)
        rope.rope_bf16(k, c, s)
        attention.attention(qr, kc, vc, np.arange(nk), query_idx=np.arange(nq))
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= 10.0 or reps == 8:
            break
    flops = attn_flops(wl.H, nq, nk) * wl.B * reps
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"fp64 NumPy oracle: rotary tables + RoPE of one {N}-token chunk's q and k, then attention "
                      f"of {nq} of its {N} queries x {wl.H} heads over {nk} keys, {reps} times; {dt:.2f} s wall; "
                      f"{len(os.sched_getaffinity(0))} host cores visible, {platform.processor() or 'cpu'}"}



_CSRC = "paper_2609_32518_amd/csrc/"
KERNEL_SOURCES = {
    "window_attn_kernel": [_CSRC + "window_attn.hip", _CSRC + "kernels.hpp", _CSRC + "seg_table.hpp"],
    "rope_append_kernel": [_CSRC + "rope_append.hip", _CSRC + "kernels.hpp", _CSRC + "seg_table.hpp"],
    "rope_norm_append_kernel": [_CSRC + "rope_append.hip", _CSRC + "kernels.hpp", _CSRC + "seg_table.hpp"],
    "copy3_kernel": [_CSRC + "copy_baseline.hip", _CSRC + "kernels.hpp"],
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_hash(kernel):
    """Hash of the kernel's sources with comments and blank space removed (a comment edit does
    not make measured counters stale; any code change does)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        text = open(os.path.join(ROOT, f)).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from profiles/traffic.json, if taken on the current kernel source."""
    try:
        rec = json.load(open(TRAFFIC_FILE))[workload][kernel]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source") != source_hash(kernel):
        return None
    return rec["bytes_per_launch"]


def profile_commands(workload="full_chunk", qknorm=False):
    """The profiling commands whose output --summarize-profile reads (run from the repo root,
    after `cd /tmp && export TMPDIR=/tmp && cd -`), DIR being their common output folder."""
    q = " --qknorm" if qknorm else ""
    b = f"python -u bench.py --workload {workload} --steps 30 --warmup 30 --no-cpu-baseline{q}"
    pmc = f"python -u bench.py --workload {workload} --steps 2 --warmup 1 --sets 1 --no-cpu-baseline{q}"
    cal = "python -u bench.py --copy-calibration 256"
    return [
        ("trace", f"rocprofv3 --kernel-trace --stats -d DIR/trace -o trace --output-format csv -- {b}"),
        ("fetch", f"rocprofv3 --pmc FETCH_SIZE -d DIR/fetch -o fetch --output-format csv -- {pmc}"),
        ("write", f"rocprofv3 --pmc WRITE_SIZE -d DIR/write -o write --output-format csv -- {pmc}"),
        ("copy_fetch", f"rocprofv3 --pmc FETCH_SIZE -d DIR/copy_fetch -o copy_fetch --output-format csv -- {cal}"),
        ("copy_write", f"rocprofv3 --pmc WRITE_SIZE -d DIR/copy_write -o copy_write --output-format csv -- {cal}"),
        ("sq", f"rocprofv3 --pmc SQ_WAVES SQ_INSTS_VALU SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_LDS "
               f"SQ_LDS_BANK_CONFLICT SQ_WAIT_INST_LDS GRBM_GUI_ACTIVE -d DIR/sq -o sq --output-format csv -- {pmc}"),
    ]


def summarize_profile(d, workload="full_chunk", qknorm=False):
    import csv
    import re
    from collections import defaultdict

    def kname(n):
        m = re.search(r"::(\w+_kernel)(<[^>]*>)?\(", n)
        if m:
            return m.group(1) + (m.group(2) or "")
        return "copy" if "copyBuffer" in n or "copy" in n.lower() else n[:40]

    def counters(name):
        per = defaultdict(lambda: defaultdict(list))
        for r in csv.DictReader(open(os.path.join(d, name, f"{name}_counter_collection.csv"))):
            per[kname(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
        return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in per.items()}

    stats = list(csv.DictReader(open(os.path.join(d, "trace", "trace_kernel_stats.csv"))))
    fetch, write = counters("fetch"), counters("write")
    cf, cw = counters("copy_fetch"), counters("copy_write")
    sq = counters("sq")
    cal_bytes = 256 * 1000 * 1000
    copy_f = max(v["FETCH_SIZE"] for k, v in cf.items() if "FETCH_SIZE" in v and v["FETCH_SIZE"] > 1000)
    copy_w = max(v["WRITE_SIZE"] for k, v in cw.items() if "WRITE_SIZE" in v and v["WRITE_SIZE"] > 1000)
    f_scale = cal_bytes / (copy_f * 1024)
    w_scale = cal_bytes / (copy_w * 1024)
    try:
        traffic = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        traffic = {}
    traffic.setdefault(workload, {})
    lines = [f"# Kernel profile — {workload} workload{' with the RMS-normalising append' if qknorm else ''}", "",
             "Commands (repo root, one MI355X, after `cd /tmp && export TMPDIR=/tmp && cd -`; DIR is an "
             "output folder; this file was written by `python bench.py --summarize-profile DIR`):", "", "```"]
    lines += [c for _, c in profile_commands(workload, qknorm)]
    lines += ["```", "", "## Kernel trace (rocprofv3 --kernel-trace --stats)", "",
              "| kernel | calls | average µs | min µs | max µs | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:6]:
        lines.append(f"| {kname(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    # the bench's own per-kernel timing launches each kernel `steps` times back to back at the
    # end of the run: the same dispatches' average, for comparison with its HIP-event figure
    trace_rows = sorted(csv.DictReader(open(os.path.join(d, "trace", "trace_kernel_trace.csv"))),
                        key=lambda r: int(r["Start_Timestamp"]))
    import synth
    wl = synth.WORKLOADS[workload]
    steps = 30 * wl.layers * wl.passes        # dispatches of the timing loop: 30 steps of the workload's calls
    attn = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace_rows
            if kname(r["Kernel_Name"]) == "window_attn_kernel"]
    if workload != "rolling" and len(attn) >= 3 * steps:
        # the trace command runs 30 warm-up steps, 30 timed steps, then 30 steps with the attention
        # between events: the latter's dispatches are what the bench's `attn` and `roofline` time
        timed = attn[2 * steps:3 * steps]
        lines.append(f"\nwindow_attn_kernel: the {steps} dispatches of the event-timed steps (the bench's `attn` "
                     f"and `roofline` figures: median of the event intervals in the step) average "
                     f"{sum(timed) / len(timed) / 1e3:.2f} µs, median {statistics.median(timed) / 1e3:.2f} µs.")
    for kern in ("window_attn_kernel", "rope_append_kernel<true>", "rope_norm_append_kernel<true, 3>", "copy3_kernel",
                 "mfma_reference_kernel"):
        durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace_rows if kname(r["Kernel_Name"]) == kern]
        if workload == "rolling" and durs:
            # the stream's bench times every call between events: its figure is the average over
            # all calls of the timed passes, which the whole-run average above approximates
            continue
        if len(durs) >= steps:
            tail = durs[-steps:]
            what = "`attn.us_per_call_back_to_back`" if kern == "window_attn_kernel" else "its figure"
            lines.append(f"\n{kern}: the last {steps} dispatches (the bench's back-to-back per-kernel timing loop, "
                         f"{what}) average {sum(tail) / len(tail) / 1e3:.2f} µs.")
    lines += ["", "## HBM traffic per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)", "",
              f"Scale factors from a plain 256 MB device copy (`--copy-calibration 256`): FETCH_SIZE read "
              f"{copy_f:.0f} KiB -> x{f_scale:.3f}; WRITE_SIZE read {copy_w:.0f} KiB -> x{w_scale:.3f}.", "",
              "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled read MB | scaled write MB | total MB |",
              "|---|---|---|---|---|---|"]
    if workload == "rolling":
        lines[-3:-2] = ["", "Per-dispatch figures here and below are averages over the stream's calls, whose "
                        "key ranges grow from 1 to 12 frames.", ""]
    for k in sorted(set(fetch) | set(write)):
        if not k.startswith(("window_attn", "attn_combine", "rope_append", "rope_norm_append", "copy3")):
            continue
        fk, wk = fetch.get(k, {}).get("FETCH_SIZE", 0.0), write.get(k, {}).get("WRITE_SIZE", 0.0)
        rb, wb = fk * 1024 * f_scale, wk * 1024 * w_scale
        lines.append(f"| {k} | {fk:.0f} | {wk:.0f} | {rb / 1e6:.2f} | {wb / 1e6:.2f} | {(rb + wb) / 1e6:.2f} |")
        base = k.split("<")[0]
        if base in KERNEL_SOURCES and (base in ("window_attn_kernel", "copy3_kernel") or k.startswith(base + "<true")):
            traffic[workload][base] = {"bytes_per_launch": round(rb + wb), "read_bytes": round(rb),
                                       "write_bytes": round(wb), "source": source_hash(base)}
    a = sq.get("window_attn_kernel")
    if a:
        # shader clock during the kernel: GPU-busy cycles of one XCD over the dispatch's duration,
        # median over the dispatches of the counter run (the first, cold one included)
        per = defaultdict(lambda: [0.0, 0])
        for r in csv.DictReader(open(os.path.join(d, "sq", "sq_counter_collection.csv"))):
            if kname(r["Kernel_Name"]) == "window_attn_kernel" and r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                per[r["Dispatch_Id"]][0] += float(r["Counter_Value"]) / 8
                per[r["Dispatch_Id"]][1] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        clocks = sorted(c / ns for c, ns in per.values() if ns > 0)
        sclk = clocks[len(clocks) // 2] if clocks else float("nan")
        cyc = a["GRBM_GUI_ACTIVE"] / 8
        tiles = a["SQ_INSTS_MFMA"] / 32
        lines += ["", "## window_attn_kernel SQ counters (per dispatch)", "",
                  f"- waves {a['SQ_WAVES']:.0f}; MFMA instructions {a['SQ_INSTS_MFMA']:.4g} "
                  f"(= 32 per wave per 64-key tile); MFMA busy cycles {a['SQ_VALU_MFMA_BUSY_CYCLES']:.4g}",
                  f"- MFMA busy fraction per SIMD {a['SQ_VALU_MFMA_BUSY_CYCLES'] / (1024 * cyc):.3f} over "
                  f"{cyc:.4g} GPU cycles (GRBM_GUI_ACTIVE / 8 XCDs)",
                  f"- shader clock during the kernel {sclk:.2f} GHz (GPU cycles per XCD / dispatch duration, "
                  f"median of {len(clocks)} dispatches: "
                  + (", ".join(f"{c:.2f}" for c in clocks) if len(clocks) <= 9 else
                     f"min {clocks[0]:.2f}, max {clocks[-1]:.2f}") + "); "
                  f"MFMA peak at that clock {1024 * 1024 * sclk / 1e3:.0f} TFLOP/s",
                  f"- non-MFMA VALU instructions per wave-tile {(a['SQ_INSTS_VALU'] - a['SQ_INSTS_MFMA']) / tiles:.1f}; "
                  f"LDS instructions per wave-tile {a['SQ_INSTS_LDS'] / tiles:.1f}; "
                  f"LDS bank conflicts {a['SQ_LDS_BANK_CONFLICT']:.0f}"]
    out = os.path.join(ROOT, "profiles", f"kernels_{workload}{'_qknorm' if qknorm else ''}.md")
    open(out, "w").write("\n".join(lines) + "\n")
    json.dump(traffic, open(TRAFFIC_FILE, "w"), indent=1, sort_keys=True)
    print("\n".join(lines))


def summarize_trace(d, name, command):
    """A kernel-time summary of one rocprofv3 --kernel-trace --stats run of any bench mode: the
    stats table and the bench's own JSON line (the last line of the run's log, DIR/run.log)."""
    import csv
    import glob
    stats_files = glob.glob(os.path.join(d, "*_kernel_stats.csv"))
    if not stats_files:
        raise SystemExit(f"no *_kernel_stats.csv under {d}")
    stats = list(csv.DictReader(open(stats_files[0])))
    lines = [f"# Kernel profile — {name}", "",
             "Command (repo root, one MI355X, after `cd /tmp && export TMPDIR=/tmp && cd -`; DIR is an output "
             "folder; this file was written by `python bench.py --summarize-trace DIR --trace-name NAME "
             "--trace-command CMD`):", "",
             "```", command, "```", "", "## rocprofv3 --stats", "",
             "| kernel | calls | average µs | min µs | max µs | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in stats[:8]:
        lines.append(f"| {r['Name'][:90]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    log = os.path.join(d, "run.log")
    if os.path.exists(log):
        last = [ln for ln in open(log).read().splitlines() if ln.startswith("{")]
        if last:
            lines += ["", "## The run's bench line", "", "```", last[-1], "```"]
    out = os.path.join(ROOT, "profiles", f"kernels_{name}.md")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_clip_profile(d, args):
    """Per-call breakdown of the last clip in a kernel trace of `bench.py --clip ...`: kernels
    grouped by the frames each layer attends to (the sampler's call sequence and the layer
    windows give the order), written to profiles/kernels_clip_<variant>.md."""
    import csv
    from collections import defaultdict

    import paper_2609_32518_amd as u
    variant, L, C, T, H = args.clip, args.layers, 3, 1560, 12
    calls = u.unstep_sampler_calls(variant, args.clip_chunks)
    n_calls = len(calls["chunk"])
    eight = set(range(1, L, 2)) if args.eight_frame_layers == "odd" else \
        set() if args.eight_frame_layers == "none" else set(range(L)) if args.eight_frame_layers == "all" else \
        {int(x) for x in args.eight_frame_layers.split(",") if x}
    sinks = [0 if variant == "self_forcing" else 2 if li in eight else 3 for li in range(L)]
    window = [C * args.clip_chunks if variant == "self_forcing" else C for _ in range(L)]
    rows = sorted(csv.DictReader(open(os.path.join(d, "clip_kernel_trace.csv"))), key=lambda r: int(r["Start_Timestamp"]))
    ours = [r for r in rows if any(k in r["Kernel_Name"] for k in ("rope_append", "window_attn", "attn_combine",
                                                                       "flow_update"))]
    fu = [i for i, r in enumerate(ours) if "flow_update" in r["Kernel_Name"]][-2 * n_calls:]
    groups = defaultdict(list)
    for c in range(n_calls):
        f0 = int(calls["start_frame"][c])
        li = -1
        for r in ours[fu[2 * c]:fu[2 * c + 1] + 1]:
            n = r["Kernel_Name"]
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            if "rope_append" in n:
                li += 1
            lo = max(0, f0 - window[max(li, 0)])
            frames = min(sinks[max(li, 0)], lo) + f0 + C - lo
            kind = ("rope_append" if "rope_append" in n else "window_attn" if "window_attn" in n else
                    "attn_combine" if "attn_combine" in n else "flow_update")
            groups[(kind, frames if kind in ("window_attn", "attn_combine") else 0)].append(dur)
    span = (int(ours[fu[-1]]["End_Timestamp"]) - int(ours[fu[0]]["Start_Timestamp"])) / 1e3
    busy = sum(sum(v) for v in groups.values())
    stats = list(csv.DictReader(open(os.path.join(d, "clip_kernel_stats.csv"))))
    cmd = (f"rocprofv3 --kernel-trace --stats -d DIR -o clip --output-format csv -- "
           f"python -u bench.py --clip {variant} --clips 2 --clip-chunks {args.clip_chunks} --layers {L} "
           f"--eight-frame-layers {args.eight_frame_layers}")
    lines = [f"# Kernel profile — whole clip, {variant} sampler", "",
             "Command (repo root, one MI355X, after `cd /tmp && export TMPDIR=/tmp && cd -`; DIR is an output "
             "folder); this file was written by `python bench.py --summarize-clip-profile DIR` with the same clip "
             "arguments:", "", "```", cmd, "```", "",
             f"Clip: {args.clip_chunks} chunks of {C} latent frames, {n_calls} DiT calls x {L} layers, "
             f"{H} heads x 128, {T} tokens per frame; eight-frame layers: {sorted(eight) if variant != 'self_forcing' else 'none'}.",
             "", "## Last clip of the trace, by kernel and attended frames", "",
             f"Span {span / 1e3:.2f} ms; kernels busy {busy / 1e3:.2f} ms ({100 * busy / span:.1f}%).", "",
             "| kernel | attended frames | launches | average µs | total ms | % of clip | TFLOP/s |",
             "|---|---|---|---|---|---|---|"]
    for (kind, fr), v in sorted(groups.items()):
        avg = sum(v) / len(v)
        tf = f"{4 * H * C * T * fr * T * 128 / (avg * 1e-6) / 1e12:.0f}" if kind == "window_attn" else ""
        lines.append(f"| {kind} | {fr or ''} | {len(v)} | {avg:.1f} | {sum(v) / 1e3:.2f} | "
                     f"{100 * sum(v) / span:.1f} | {tf} |")
    lines += ["", "## rocprofv3 --stats (whole run: warm-up and timed clips)", "",
              "| kernel | calls | average µs | % of GPU time |", "|---|---|---|---|"]
    for r in stats[:8]:
        lines.append(f"| {r['Name'][:90]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.1f} |")
    out = os.path.join(ROOT, "profiles", f"kernels_clip_{variant}.md")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def oproj_bench(u, torch, args):
    """The output projection of the full-frame chunk's attention output ([4680, 12 x 128] x
    [1536, 1536]^T + bias, bf16) over rotating inputs, HIP events around back-to-back calls;
    then the V/O truncated SVD of one 1536 x 1536 float32 weight at rank 1413 (init time)."""
    dev = "cuda"
    M, N, K = 4680, 1536, 1536
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    xs = [torch.randn((M, K), generator=g, device=dev).to(torch.bfloat16) for _ in range(16)]   # 230 MB
    w32 = torch.randn((N, K), generator=g, device=dev) / math.sqrt(K)
    b = torch.randn((N,), generator=g, device=dev).to(torch.bfloat16)
    r = 1413                     # the paper's V/O rank: round(0.92 * 1536) (App. A.4)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, w, _ = u.unstep_svd_truncate(w32, r)
    svd_ms = (time.perf_counter() - t0) * 1e3
    t0 = time.perf_counter()
    u.unstep_svd_truncate(w32, r)
    svd_ms2 = (time.perf_counter() - t0) * 1e3
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    for k in range(max(args.warmup, 20)):
        u.unstep_linear(xs[k % 16], w, b, out=y)
    n = max(args.steps, 100)
    it = [0]

    def call():
        u.unstep_linear(xs[it[0] % 16], w, b, out=y)
        it[0] += 1

    # kernel time: behind the device-side spin (the binding's host time per call is comparable to
    # the kernel's, so back-to-back calls alone would time the host); then the same calls without
    # the spin, the rate a Python caller gets
    us = timed_passes(torch, call, n, spin=True, batch=50) * 1e3
    us_host = timed_passes(torch, call, n, spin=False) * 1e3
    flops = 2.0 * M * N * K
    tf = flops / (us * 1e-6) / 1e12
    print(json.dumps({"metric": "output projection µs per chunk (4680 x 1536 x 1536 bf16 + bias)",
                      "value": round(us, 2), "unit": "us", "higher_is_better": False, "calls": n,
                      "us_per_call_back_to_back_through_binding": round(us_host, 2),
                      "tflops": round(tf, 1), "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                      "svd_truncate_ms": {"first_call": round(svd_ms, 1), "second_call": round(svd_ms2, 1),
                                          "shape": [N, K], "rank": r},
                      "config": {"M": M, "N": N, "K": K, "bias": True}, "dtype": "bf16, fp32 accumulate",
                      "data": "synthetic"}), flush=True)


def flow_update_bench(u, torch, args):
    """Renoise (Equation 1) then emit (Equation 3) at the clean-cache level on a chunk's latent,
    over rotating buffer sets; per-op time from HIP events around back-to-back launches."""
    shape = (1, 16, 3, 60, 104)
    n = math.prod(shape)
    g = torch.Generator(device="cuda")
    sets = []
    for i in range(max(args.sets, 64)):          # ~115 MB: beyond the reuse of one set in L2
        g.manual_seed(100 + i)
        mk = lambda: torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16)
        sets.append((mk(), mk(), mk(), torch.empty(shape, dtype=torch.bfloat16, device="cuda")))
    sigma = 0.02

    def run(k):
        x, e, v, o = sets[k % len(sets)]
        u.unstep_renoise(x, e, sigma, out=o)
        u.unstep_emit(o, v, sigma, out=o)

    for k in range(args.warmup):
        run(k)
    it = [0]

    def pair():
        run(it[0])
        it[0] += 1

    # kernel time behind the device-side spin (a pair's host time through the binding is several
    # times its GPU time), then the rate of back-to-back calls from Python
    us_pair = timed_passes(torch, pair, args.steps, spin=True, batch=64) * 1e3
    us_host = timed_passes(torch, pair, args.steps, spin=False) * 1e3
    nbytes = 2 * 3 * 2 * n                       # two ops, each reads two bf16 tensors and writes one
    print(json.dumps({"metric": "clean-cache renoise + emit µs per chunk latent", "value": round(us_pair, 3),
                      "unit": "us", "higher_is_better": False, "steps": args.steps, "warmup": args.warmup,
                      "us_per_pair_back_to_back_through_binding": round(us_host, 3),
                      "bytes": nbytes, "gbs": round(nbytes / (us_pair * 1e-6) / 1e9, 1),
                      "hbm_frac": round(nbytes / (us_pair * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                      "config": {"latent": list(shape), "sigma": sigma}, "dtype": "bf16 in/out, f64 math",
                      "data": "synthetic"}), flush=True)


def clip_bench(u, torch, args):
    """Whole clips at the paper's shapes: for every DiT call of the sampler, renoise the chunk's
    latent, run one chunk step (RoPE + KV append + windowed attention) in each of the layers,
    each layer with its own cache (nine frames: 3 sinks + 6 recent; eight frames: 2 + 6; the
    original sampler: every frame), then emit.  Synthetic q/k/v, noise and velocities are drawn
    up front and rotated; the rotary tables of each start frame are built once, on a side stream
    while the compute stream runs earlier calls, and cached for the process (so the timed clips
    find them built).  Caches start empty for each clip."""
    dev = "cuda"
    H, GH, GW, C = 12, 30, 52, 3
    T = GH * GW
    N = C * T
    L, n_chunks = args.layers, args.clip_chunks
    if args.eight_frame_layers == "none":
        eight = set()
    elif args.eight_frame_layers == "all":
        eight = set(range(L))
    elif args.eight_frame_layers == "odd":
        eight = set(range(1, L, 2))
    else:
        eight = {int(x) for x in args.eight_frame_layers.split(",") if x}
    if args.clip == "self_forcing":
        windows = [(0, C * n_chunks, C * n_chunks)] * L            # every frame kept
    else:
        windows = [((2 if li in eight else 3), C, 2 * C) for li in range(L)]   # (S, W, R)
    calls = u.unstep_sampler_calls(args.clip, n_chunks)
    n_calls = len(calls["chunk"])

    g = torch.Generator(device=dev)

    def randn(shape, seed):
        g.manual_seed(seed)
        return torch.randn(shape, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)

    pool = [tuple(randn((1, N, H, 128), 50 + 3 * i + j) for j in range(3)) for i in range(8)]   # 345 MB
    latent = (1, 16, C, 2 * GH, 2 * GW)
    noise = [randn(latent, 900 + i) for i in range(8)]
    vel = [randn(latent, 950 + i) for i in range(8)]
    x = randn(latent, 999)
    q_rot = torch.empty((1, N, H, 128), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q_rot)
    bufs = []
    for (S, W, R) in windows:
        rows = (S + R) * T
        bufs.append((torch.zeros((1, H, rows, 128), dtype=torch.bfloat16, device=dev),
                     torch.zeros((1, H, rows, 128), dtype=torch.bfloat16, device=dev)))
    side = torch.cuda.Stream()                                     # default priority
    compute = torch.cuda.current_stream()

    def new_caches():
        return [u.Cache(1, H, GH, GW, S, R, device=dev, k_cache=k, v_cache=v)
                for (S, W, R), (k, v) in zip(windows, bufs)]

    # one workspace for every layer and call (the calls run in stream order)
    probe = new_caches()
    ws_need = max(probe[li].workspace_bytes(int(f0), C, windows[li][1])
                  for li in range(L) for f0 in set(calls["start_frame"].tolist()))
    ws = torch.empty(max(ws_need, 1), dtype=torch.uint8, device=dev)
    del probe

    flops = 0.0
    for ci in range(n_calls):
        f0 = int(calls["start_frame"][ci])
        for (S, W, R) in windows:
            lo = max(0, f0 - W)
            keys = (min(S, lo) + (f0 + C - lo)) * T
            flops += attn_flops(H, N, keys)

    # rotary tables are cached per start frame for the process (built during the warm-up clip)
    tables = {}

    def run_clip(xt_buf):
        caches = new_caches()
        k = 0
        for ci in range(n_calls):
            f0 = int(calls["start_frame"][ci])
            sigma = float(calls["sigma"][ci])
            if f0 not in tables:
                with torch.cuda.stream(side):
                    tables[f0] = u.unstep_rope_tables(f0, C, GH, GW, stream=side)
            cos_t, sin_t = tables[f0]
            u.unstep_renoise(x, noise[ci % 8], sigma, out=xt_buf)
            for li, cache in enumerate(caches):
                q, kk, v = pool[k % len(pool)]
                k += 1
                cache.unstep_step(f0, C, windows[li][1], q, kk, v, cos_t, sin_t, q_rot=q_rot, out=out,
                                  workspace=ws)
            u.unstep_emit(xt_buf, vel[ci % 8], sigma, out=x)
        return caches

    xt_buf = torch.empty_like(x)
    for _ in range(max(1, args.warmup_clips)):
        run_clip(xt_buf)
    torch.cuda.synchronize()
    clips = max(1, args.clips)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(compute)
    for _ in range(clips):
        run_clip(xt_buf)
    e1.record(compute)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / clips
    ms = e0.elapsed_time(e1) / clips
    latent_frames = C * n_chunks
    video_frames = 1 + 4 * (latent_frames - 1)
    tf = flops / (ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": "attention path ms per clip (sampler calls x layers: RoPE + KV append + windowed attention, "
                  "renoise, emit)",
        "value": round(ms, 3), "unit": "ms", "higher_is_better": False, "clips": clips,
        "wall_ms_per_clip": round(wall * 1e3, 3), "dit_calls": n_calls, "layer_steps": n_calls * L,
        "us_per_layer_step": round(ms * 1e3 / (n_calls * L), 2),
        "attn_tflops": round(tf, 1), "attn_frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4),
        "video_frames_per_s_attention_path_only": round(video_frames / (ms * 1e-3), 1),
        "config": {"workload": f"clip_{args.clip}", "chunks": n_chunks, "latent_frames": latent_frames,
                   "video_frames": video_frames, "layers": L, "eight_frame_layers": sorted(eight)
                   if args.clip != "self_forcing" else [], "heads": H, "grid": [GH, GW], "chunk_frames": C},
        "dtype": "bf16 in, fp32 accumulate", "data": "synthetic"}), flush=True)


SUB_WORKLOADS = ("tiny", "unwindowed", "short_refine", "rolling", "paper_default")


def mfma_reference_us(u, torch, groups, waves_per_simd, mfmas, launches):
    """µs per launch of unstep_mfma_reference in this shape on seeded N(0, 1) bf16 operands,
    launched back to back (behind the device-side spin when a launch is short)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(41)
    src = torch.randn(groups * 512 * 128, generator=g, device="cuda").to(torch.bfloat16)
    out = torch.empty((groups, 8), dtype=torch.float32, device="cuda")
    ms = timed_passes(torch, lambda: u.unstep_mfma_reference(src, groups, waves_per_simd, mfmas, out=out), launches,
                      spin=mfmas < 8192, batch=128)
    return ms * 1e3


def mfma_reference_bench(u, torch, args):
    """The MFMA rate reference in the launch shapes of the full-frame chunk's attention (228
    work-groups, two multiplying waves per SIMD, 32 MFMAs per key tile plus one M phase: 9408
    per wave) and of its output projection (228 work-groups, one multiplying wave per SIMD, 768
    MFMAs per wave)."""
    steps = max(args.steps, 30)
    shapes = {"attention_full_chunk": (228, 2, 32 * (293 + 1)), "projection_4680x1536x1536": (228, 1, 768)}
    res = {"metric": "MFMA-only µs per launch on random bf16 operands", "unit": "us", "higher_is_better": False,
           "launches": steps, "shapes": {}}
    for name, (groups, wps, mfmas) in shapes.items():
        us = mfma_reference_us(u, torch, groups, wps, mfmas, steps)
        flops = groups * 4 * wps * mfmas * 32 * 32 * 16 * 2
        res["shapes"][name] = {"groups": groups, "waves_per_simd": wps, "mfmas_per_wave": mfmas,
                               "us_per_call": round(us, 2), "tflops": round(flops / (us * 1e-6) / 1e12, 1)}
    print(json.dumps(res), flush=True)


def measure_workload(u, torch, wl, n_sets, steps, warmup, qknorm=False, no_split=False):
    """Time `steps` whole steps of a workload after `warmup` untimed ones, then each kernel of the
    step on its own; returns the figures of one bench record (attention and append per call,
    with their roofline fractions, and the step)."""
    plan = Plan(u, torch, wl, n_sets, qknorm=qknorm, no_split=no_split)
    flops, _ = plan.per_step()
    torch.cuda.synchronize()
    for _ in range(warmup):
        plan.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        plan.step()
    t_enq = time.perf_counter() - t0
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms = dt * 1e3 / steps

    # the same steps again with each call's attention between two HIP events on its stream, so
    # that the attention kernel's duration is measured in the step as it runs (after the append
    # pass, which on this power-limited chip changes the clock the attention runs at).  The
    # events are left out of the timed steps above (each adds a short gap to the stream), and
    # the figure is the median over the steps: a pair that brackets a moment when the host fell
    # behind includes the idle time
    events = []
    for _ in range(steps):
        plan.step(attn_events=events)
    torch.cuda.synchronize()
    ncalls_step = len(plan.calls)
    in_step = [e0.elapsed_time(e1) for e0, e1 in events]
    per_call_ms = [statistics.median(in_step[c::ncalls_step]) for c in range(ncalls_step)]
    att_ms = sum(per_call_ms)

    # then each kernel of the step on its own, launched `steps` times back to back (same calls,
    # same rotating buffer sets) between two HIP events on the stream it runs on
    extra = {}
    if wl.name == "rolling":
        app_ms, att = plan.time_rolling(steps)
        nc = len(plan.calls)
        att_b2b_ms = sum(att) / steps
        per_chunk = [x * 1e3 for x in per_call_ms]
        extra["attn_per_chunk_us"] = {"mean": round(sum(per_chunk) / nc, 2), "max": round(max(per_chunk), 2),
                                      "min": round(min(per_chunk), 2),
                                      "steady_12_frames_mean": round(sum(per_chunk[11:]) / len(per_chunk[11:]), 2)}
    else:
        app_ms, att_b2b_ms = plan.time_kernels(steps)
    per_call_flops = sum(attn_flops(wl.H, C * wl.T, plan.keys(f0, C, W)) * wl.B for (_, f0, C, W) in plan.calls)
    per_call_bytes = sum(plan.append_bytes(C) for (_, f0, C, W) in plan.calls)
    ncalls = len(plan.calls)
    attn_us = att_ms * 1e3 / ncalls
    app_us = app_ms * 1e3 / ncalls
    attn_tflops = per_call_flops / (att_ms * 1e-3) / 1e12
    rope_gbs = per_call_bytes / (app_ms * 1e-3) / 1e9
    if ncalls > 1:
        extra["attn_us_per_step"] = round(att_ms * 1e3, 1)
    # the bandwidth reference: q, k, v copied into three buffers in one launch per call
    copy_ms = plan.time_copy_baseline(steps)
    copy_bytes = sum(6 * 2 * wl.B * C * wl.T * wl.H * 128 for (_, f0, C, W) in plan.calls)
    copy_gbs = copy_bytes / (copy_ms * 1e-3) / 1e9
    extra["append_copy_baseline"] = {"kernel": "copy3", "us_per_call": round(copy_ms * 1e3 / ncalls, 2),
                                     "bytes_per_call": copy_bytes // ncalls, "gbs": round(copy_gbs, 1),
                                     "frac": round(copy_gbs / PEAK_HBM_GBS, 4),
                                     "traffic": measured_traffic("copy3_kernel", wl.name)}
    # the MFMA work alone of this attention launch shape, on random bf16 operands (the chip's
    # clock depends on the data): what the kernel's time compares with before the published peak
    if wl.name != "rolling":
        (_, f0, C, W) = plan.calls[0]
        groups, mfmas = plan.attn_launch_shape(f0, C, W)
        ref_us = mfma_reference_us(u, torch, groups, 2, mfmas, steps)
        extra["mfma_reference"] = {"kernel": "mfma_reference", "groups": groups, "waves_per_simd": 2,
                                   "mfmas_per_wave": mfmas, "us_per_call": round(ref_us, 2),
                                   "attn_time_over_reference": round(attn_us / ref_us, 4)}
    app_kernel = "rope_norm_append_kernel" if qknorm else "rope_append_kernel"
    rec = {
        "value": round(flops / (ms * 1e-3) / 1e12, 3),
        "ms_per_step": round(ms, 5),
        "us_per_step": round(ms * 1e3, 2),
        "host_enqueue_us_per_step": round(t_enq * 1e6 / steps, 2),
        "steps": steps, "warmup": warmup,
        "config": {"workload": wl.name, "batch": wl.B, "heads": wl.H, "head_dim": 128,
                   "grid": [wl.grid_h, wl.grid_w], "chunk_frames": wl.C, "sink_frames": wl.S,
                   "window_frames": wl.W, "ring_frames": wl.R, "queries": wl.n_query,
                   "keys": plan.keys(wl.f0, wl.C, wl.W), "calls_per_step": ncalls,
                   "buffer_sets": len(plan.sets)},
        "attn": {"kernel": "window_attn", "us_per_call": round(attn_us, 2), "tflops": round(attn_tflops, 2),
                 "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                 "us_per_call_back_to_back": round(att_b2b_ms * 1e3 / ncalls, 2),
                 "traffic": measured_traffic("window_attn_kernel", wl.name)},
        "rope_append": {"kernel": app_kernel[:-len("_kernel")], "us_per_call": round(app_us, 2),
                        "gbs": round(rope_gbs, 1), "frac": round(rope_gbs / PEAK_HBM_GBS, 4),
                        "traffic": measured_traffic(app_kernel, wl.name)},
    }
    rec.update(extra)
    del plan
    return rec


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(args.summarize_profile, args.workload or "full_chunk", args.qknorm)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.trace_name or "trace", args.trace_command or "")
        return
    if args.summarize_clip_profile:
        summarize_clip_profile(args.summarize_clip_profile, args)
        return
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (the step shards by head across GPUs, but no "
              f"multi-GPU path is built); got --gpus {args.gpus}", file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        n = args.copy_calibration * 1000 * 1000
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 5}), flush=True)
        return
    import paper_2609_32518_amd as u

    if args.flow_update:
        flow_update_bench(u, torch, args)
        return
    if args.clip:
        clip_bench(u, torch, args)
        return
    if args.oproj:
        oproj_bench(u, torch, args)
        return
    if args.mfma_reference:
        mfma_reference_bench(u, torch, args)
        return
    headline = args.workload or "full_chunk"
    wl = synth.WORKLOADS[headline]
    m = measure_workload(u, torch, wl, args.sets, args.steps, args.warmup, qknorm=args.qknorm,
                         no_split=args.no_split)
    app_kernel = "rope_norm_append_kernel" if args.qknorm else "rope_append_kernel"
    res = {
        "metric": METRIC, "value": m["value"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": m["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": dict(m["config"], qk_rmsnorm=bool(args.qknorm), parallelism="single GPU"),
        "us_per_step": m["us_per_step"],
        "host_enqueue_us_per_step": m["host_enqueue_us_per_step"],
        "attn": m["attn"],
        "rope_append": m["rope_append"],
        "roofline": {"bound": "mfma", "achieved": m["attn"]["tflops"], "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": m["attn"]["frac"],
                     "traffic": measured_traffic("window_attn_kernel", wl.name)},
        "rope_roofline": {"bound": "hbm", "achieved": m["rope_append"]["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                          "frac": m["rope_append"]["frac"],
                          "traffic": measured_traffic(app_kernel, wl.name)},
    }
    for k in ("attn_per_chunk_us", "attn_us_per_step", "append_copy_baseline", "mfma_reference"):
        if k in m:
            res[k] = m[k]
    # every other workload of the benchmark, measured in the same run (same box, same clock
    # conditions), with fewer steps: each a full step of its own shape
    if args.workload is None and not args.qknorm and args.sub_steps > 0:
        res["workloads"] = {}
        for name in SUB_WORKLOADS:
            sub = measure_workload(u, torch, synth.WORKLOADS[name], args.sets, args.sub_steps, args.sub_warmup)
            sub.pop("config")
            res["workloads"][name] = sub
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, args.cpu_queries)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
