"""The C ABI from C: tests/c_abi/host_client.c, a C99 program that includes include/unstep.h
and links libunstep.so, is compiled with the system C compiler (warnings as errors) and run.
It calls only the entry points that touch no device memory and checks tables, the cache
index and the sampler's call sequence against closed forms and the paper's counts."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_32518_amd")
LIB = os.path.join(PKG, "libunstep.so")


def test_c_client_compiles_links_and_passes(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(LIB):
        pytest.skip("libunstep.so not built")
    exe = str(tmp_path / "host_client")
    build = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", f"-I{os.path.join(ROOT, 'include')}",
                            os.path.join(ROOT, "tests", "c_abi", "host_client.c"), f"-L{PKG}", "-lunstep",
                            f"-Wl,-rpath,{PKG}", "-lm", "-o", exe], capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stderr + run.stdout
    assert "ok" in run.stdout
