"""The C ABI from a plain C99 client: tests/c/abi_check.c compiles with gcc
(-std=c99 -pedantic -Werror) against include/headcast.h, links libheadcast.so
and runs the host-only entry points (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2607_20125_amd")
LIB = os.path.join(LIB_DIR, "libheadcast.so")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_client_builds_and_runs(tmp_path):
    if not os.path.exists(LIB):
        pytest.fail("libheadcast.so is not built (run __graft_entry__.build())")
    exe = tmp_path / "abi_check"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_check.c"),
           "-L", LIB_DIR, "-lheadcast", f"-Wl,-rpath,{LIB_DIR}", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "abi_check: ok" in run.stdout
