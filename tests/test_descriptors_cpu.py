"""The library's launch descriptors checked on the CPU, under AddressSanitizer and
UndefinedBehaviorSanitizer, against the oracle's cache model (paper Section 3.1 and
Appendix A.5: the positions are host integers; Section 3.3 and Appendix A.3: the retained
window).

tests/c_abi/record_launch.cpp links the library's host sources (the C ABI, the attention work
split, the rotary tables) with launchers that record the kernel descriptors instead of
launching them.  For each call it reports the slot every appended frame is written to and, for
attention, the cache row the K and V loaders fetch for every retained key of every query tile,
computed with the kernels' own address arithmetic (seg_table.hpp) over each work-group's
segments and loader cursors, plus coverage, bounds and merge checks.  Here those rows must equal
the oracle's slot map and key rows, call by call, over the seeded random call sequences of the
GPU suite and the benchmark workloads.  No GPU is used.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest

import synth
from oracle.kvcache import KVCacheOracle, OracleError, slot_of_frame
from tests.gpu_helpers import random_medium_cases, random_shape_cases

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32518_amd", "csrc")
BIN = os.path.join(ROOT, "_build", "record_launch")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

RC = {"shape": -2, "range": -3, "state": -4}


@pytest.fixture(scope="module")
def driver():
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime.h")):
        pytest.skip("needs g++ and the HIP headers")
    os.makedirs(os.path.dirname(BIN), exist_ok=True)
    # host code only: g++, no .hip source on this line; the sanitizers instrument the library's
    # host sources and the driver
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include",
           f"-I{CSRC}", os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "attn_plan.cpp"),
           os.path.join(CSRC, "rope_tables.cpp"), os.path.join(ROOT, "tests", "c_abi", "record_launch.cpp"),
           "-o", BIN]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return BIN


def run(driver, script):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([driver], input="\n".join(script) + "\n", capture_output=True, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    return [json.loads(l) for l in r.stdout.splitlines()]


class Replay:
    """The oracle's side of a call script: expected status, frame map, append slots and key rows."""

    def __init__(self, B, H, gh, gw, S, R):
        self.o = KVCacheOracle(B, H, 128, gh, gw, S, R)
        self.B, self.H, self.T = B, H, gh * gw
        self.script = [f"create {B} {H} {gh} {gw} {S} {R}"]
        self.expect = [dict(rc=0, append=[], attn=[])]

    def _zeros(self, C):
        return np.zeros((self.B, C * self.T, self.H, 128), np.uint16)

    def append(self, f0, C, with_q=False, advance=False):
        self.script.append(f"advance {f0} {C}" if advance else f"append {f0} {C} {int(with_q)}")
        try:
            self.o.append(f0, C, self._zeros(C), self._zeros(C))
            slots = [slot_of_frame(f, self.o.S, self.o.R) for f in range(f0, f0 + C)]
            self.expect.append(dict(rc=0, append=[] if advance else [slots], attn=[]))
        except OracleError as e:
            self.expect.append(dict(rc=RC[e.kind], append=[], attn=[]))

    def attn(self, f0, C, W, kind="attn", split=True):
        self.script.append(f"noalloc {f0} {C} {W}" if kind == "noalloc" else f"{kind} {f0} {C} {W} {int(split)}")
        try:
            self.expect.append(dict(rc=0, append=[], attn=[self.o.key_rows(f0, C, W).tolist()]))
        except OracleError as e:
            self.expect.append(dict(rc=RC[e.kind], append=[], attn=[]))

    def step(self, f0, C, W, split=True):
        self.script.append(f"step {f0} {C} {W} {int(split)}")
        import copy
        trial = copy.deepcopy(self.o)
        try:
            trial.append(f0, C, self._zeros(C), self._zeros(C))
            rows = trial.key_rows(f0, C, W).tolist()
        except OracleError as e:
            self.expect.append(dict(rc=RC[e.kind], append=[], attn=[]))
            return
        self.o = trial
        slots = [slot_of_frame(f, self.o.S, self.o.R) for f in range(f0, f0 + C)]
        self.expect.append(dict(rc=0, append=[slots], attn=[rows]))

    def check(self, out, what):
        assert len(out) == len(self.expect), what
        for i, (got, want) in enumerate(zip(out, self.expect)):
            where = f"{what}: call {i} `{self.script[i]}`"
            assert got["rc"] == want["rc"], (where, got["rc"], want["rc"])
            assert [a["slots"] for a in got["append"]] == want["append"], where
            for a in got["append"]:
                assert a["in_bounds"], where
            assert len(got["attn"]) == len(want["attn"]), where
            for a, rows in zip(got["attn"], want["attn"]):
                for flag in ("covered_once", "k_v_agree", "same_rows_every_tile", "rows_in_bounds", "tail_rows_ok",
                             "merge_reads_written", "single_run_tiles_ok"):
                    assert a[flag], (where, flag)
                assert a["n_keys"] == len(rows), where
                # the launch walks the retained rows in ascending cache order (attention over
                # the retained set does not depend on the order of its keys)
                assert a["rows"] == sorted(rows), where
        # the frame map after the last call
        assert out[-1]["frame_of_slot"] == self.o.frame_of_slot and out[-1]["newest"] == self.o.newest, what


def test_driver_reports_a_planted_slot_mistake(driver):
    # the comparison is not vacuous: the oracle's rows shifted by one row must not match
    r = Replay(1, 1, 2, 3, 0, 4)
    r.append(0, 2)
    r.attn(0, 2, 0)
    out = run(driver, r.script)
    r.check(out, "as is")
    r.expect[-1]["attn"][0] = [x + 1 for x in r.expect[-1]["attn"][0]]
    with pytest.raises(AssertionError):
        r.check(out, "planted")


@pytest.mark.parametrize("cases", ["small", "medium"])
def test_random_call_sequences_match_the_oracle(driver, cases):
    # the GPU suite's seeded random shapes and call sequences, each call also attended through the
    # workspace-free and the allocation-free entry points, with re-appends and failing calls
    specs = random_shape_cases() if cases == "small" else random_medium_cases()
    rng = np.random.default_rng(11 if cases == "small" else 12)
    for n, c in enumerate(specs):
        r = Replay(c["B"], c["H"], c["gh"], c["gw"], c["S"], c["R"])
        for (f0, split, _) in c["calls"]:
            r.step(f0, c["C"], c["W"], split)
            r.attn(f0, c["C"], c["W"], "attn", not split)
            r.attn(f0, c["C"], c["W"], "noalloc")
            if rng.random() < 0.2:                       # a window wider than the ring allows
                r.attn(f0, c["C"], c["W"] + c["R"] + 1)
            if rng.random() < 0.2:                       # a gap
                r.append(f0 + 2 * c["C"] + 1, c["C"])
        out = run(driver, r.script)
        r.check(out, f"{cases} case {n}")


@pytest.mark.parametrize("name", ["tiny", "full_chunk", "unwindowed", "short_refine", "rolling", "paper_default"])
def test_benchmark_workloads_match_the_oracle(driver, name):
    wl = synth.WORKLOADS[name]
    r = Replay(wl.B, wl.H, wl.grid_h, wl.grid_w, wl.S, wl.R)
    if name == "rolling":
        for c in range(wl.chunks):
            r.step(c, 1, wl.W, split=True)
    else:
        for f0 in range(0, wl.f0, wl.C):
            r.append(f0, wl.C, advance=(f0 + wl.C <= wl.f0 - wl.W))
        for p in range(wl.passes):
            r.step(wl.f0, wl.C, wl.W, split=True)
        r.attn(wl.f0, wl.C, wl.W, "attn", split=False)
        r.attn(wl.f0, wl.C, wl.W, "noalloc")
    out = run(driver, r.script)
    r.check(out, name)
