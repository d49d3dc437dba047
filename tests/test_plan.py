"""Invariants of the host-side tail balancing of dense launches
(paper_2607_20125_amd/csrc/hc_plan.h): tests/c/plan_check.cpp builds work lists
shaped like the runtime's, balances them for several device sizes and checks
that every unit's keys are covered exactly once in whole tiles, that partial
slots and merge items stay consistent (at most 32 slots per item), that runs
keep one length per XCD, and that the simulated end time never grows."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_tail_balancing_invariants(tmp_path):
    exe = tmp_path / "plan_check"
    cmd = ["g++", "-std=c++17", "-O1", "-Wall", "-Wextra", "-Werror",
           "-I", os.path.join(ROOT, "paper_2607_20125_amd", "csrc"),
           os.path.join(ROOT, "tests", "c", "plan_check.cpp"), "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "plan_check: ok" in run.stdout
