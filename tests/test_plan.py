"""Invariants of the host-side planning of dense launches
(paper_2607_20125_amd/csrc/hc_plan.h), compiled from tests/c/plan_check.cpp:

* tail balancing: work lists built by the runtime's planner are balanced for
  several device sizes; every unit's keys are covered exactly once in whole
  tiles, partial slots and merge items stay consistent (at most 32 slots per
  item), runs keep one length per XCD, and the simulated end time never grows;
* key ranges: for every L that is a multiple of 8 up to 4096 and every window
  of 2 to 32 blocks, with one and two Sink-Dummy slots, before and after
  balancing, and for the classification sweep and cells of 2 to 12 positions,
  every unit's whole-tile reads end inside its head's part of the buffer whose
  size the runtime allocates (a buffer without the spare tile at the end of
  each head fails this)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_tail_balancing_invariants(tmp_path):
    exe = tmp_path / "plan_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
           # address and undefined-behaviour checks on the host planner / layout code
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "paper_2607_20125_amd", "csrc"),
           os.path.join(ROOT, "tests", "c", "plan_check.cpp"), "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "plan_check: ok" in run.stdout
