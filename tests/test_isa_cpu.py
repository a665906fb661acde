"""The compiled gfx950 assembly of the kernels that issue direct-to-LDS loads as inline assembly.

A vector-memory instruction that reads an SGPR which a VALU instruction wrote (v_readfirstlane,
v_readlane, a compare into an SGPR pair) needs 5 wait states between the two on this GPU family;
with fewer, the load may take the register's previous contents as its address.  The compiler
inserts those wait states before the memory instructions it generates itself, but it does not
know what an inline-assembly string does, so nothing guarantees them before the attention and
projection kernels' `global_load_lds_dwordx4`.  This test compiles both sources exactly as the
build does and checks every such load: within the 5 wait states before it (each instruction one,
`s_nop n` n + 1) no VALU instruction writes an SGPR of its scalar base, and that window does not
start in another basic block (where the predecessor's last instructions could not be checked).
CPU only: hipcc cross-compiles for gfx950 without a GPU.
"""
import importlib.util
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32518_amd", "csrc")
WAIT_STATES = 5


def _build_module():
    spec = importlib.util.spec_from_file_location("unstep_build", os.path.join(ROOT, "paper_2609_32518_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _assembly(source: str) -> str:
    b = _build_module()
    try:
        cc = b.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not found")
    r = subprocess.run([cc] + b.COMMON + b.DEVICE + ["--cuda-device-only", "-S", os.path.join(CSRC, source), "-o", "-"],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    return r.stdout


def _sgprs(tok: str) -> set:
    m = re.match(r"s\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok)
    return {int(m.group(1))} if m else set()


# VALU instructions with a scalar destination besides (or instead of) a vector one in the second
# operand: carry-out and scale-flag forms
_SDST_SECOND = re.compile(r"v_(add_co|sub_co|subrev_co|addc_co|subb_co|subbrev_co|div_scale|mad_u64_u32|mad_i64_i32)")


def _valu_sgpr_writes(words) -> set:
    """SGPRs a VALU instruction (mnemonic, operands...) writes: its destination, and the second
    operand of the carry-out forms."""
    out = _sgprs(words[1]) if len(words) > 1 else set()
    if _SDST_SECOND.match(words[0]) and len(words) > 2:
        out |= _sgprs(words[2])
    return out


def scan(asm: str):
    """(loads, problems): problems lists the loads whose base may be read too early."""
    lines = asm.splitlines()
    loads, problems = 0, []
    for i, line in enumerate(lines):
        m = re.search(r"global_load_lds_dwordx4\s+v\d+,\s*(s\[\d+:\d+\])", line)
        if not m:
            continue
        loads += 1
        base = _sgprs(m.group(1))
        waits = 0
        for j in range(i - 1, -1, -1):
            t = lines[j].strip()
            if not t or t.startswith(";") or (t.startswith(".") and not t.endswith(":")):
                continue                                   # comments, directives
            if t.endswith(":"):
                problems.append(f"line {i + 1}: only {waits} wait states in its block before the load")
                break
            words = t.replace(",", " ").split()
            if words[0].startswith("v_") and _valu_sgpr_writes(words) & base:
                problems.append(f"line {i + 1}: base {m.group(1)} written by `{t}` {waits} wait states before")
                break
            nop = re.match(r"s_nop\s+(\d+)", t)
            waits += int(nop.group(1)) + 1 if nop else 1
            if waits >= WAIT_STATES:
                break
    return loads, problems


def test_scan_finds_a_planted_hazard():
    """The checker itself: a VALU write of the base right before the load is reported, and
    s_nop 4 in between clears it."""
    planted = "\n".join(["k:", "\ts_mov_b32 s4, 0", "\ts_mov_b32 s5, 0", "\ts_mov_b32 s6, 0", "\ts_mov_b32 s7, 0",
                         "\tv_readfirstlane_b32 s3, v5", "\tv_readfirstlane_b32 s2, v4",
                         "\t;;#ASMSTART", "\tglobal_load_lds_dwordx4 v1, s[2:3]", "\t;;#ASMEND"])
    assert scan(planted)[0] == 1 and len(scan(planted)[1]) == 1
    fixed = planted.replace("\t;;#ASMSTART", "\t;;#ASMSTART\n\ts_nop 4")
    assert scan(fixed) == (1, [])
    other = planted.replace("s3, v5", "s9, v5").replace("s2, v4", "s8, v4")
    assert scan(other) == (1, [])
    carry = planted.replace("\tv_readfirstlane_b32 s2, v4", "\tv_add_co_u32_e64 v9, s[2:3], v4, v5")
    assert len(scan(carry)[1]) == 1
    at_block_start = "\n".join(["k:", "\tglobal_load_lds_dwordx4 v1, s[2:3]"])
    assert len(scan(at_block_start)[1]) == 1


@pytest.mark.parametrize("source", ["window_attn.hip", "linear.hip"])
def test_inline_asm_loads_read_no_freshly_written_sgpr(source):
    loads, problems = scan(_assembly(source))
    assert loads > 0, "no direct-to-LDS load found: the scan no longer matches the kernel"
    assert not problems, "\n".join(problems[:20])
