"""Invariants of the Spatial path's layout and tiling
(paper_2607_20125_amd/csrc/hc_geometry.h): tests/c/geometry_check.cpp checks, for
every grid up to 40 x 72 and radii up to 12, that the column tiles cover each frame
column once and their halo columns hold every query's column window, that the live
steps of every row tile hold every window row and only steps with rows inside the
frame, and that every read stays within rows_per_step - 1 rows of its frame (the
buffer's leading and trailing keys cover the outermost frames) with column groups
clamped into the row, and that the key-frame split rule picks the documented range
counts for the Wan-shaped grids and stays within its bounds."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_spatial_layout_invariants(tmp_path):
    exe = tmp_path / "geometry_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
           # address and undefined-behaviour checks on the host planner / layout code
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "paper_2607_20125_amd", "csrc"),
           "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "geometry_check.cpp"), "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "geometry_check: ok" in run.stdout
