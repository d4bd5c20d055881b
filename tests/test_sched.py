"""The kernels' tile-schedule arithmetic (paper_2608_00029_amd/csrc/attn_sched.h),
compiled with the host C++ compiler and checked exhaustively over sequence
lengths, tiles and waves (tests/sched_check.cpp)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_ring_waits_and_buffer_reuse(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "sched_check")
    subprocess.run([cxx, "-std=c++17", "-O1", "-I", os.path.join(ROOT, "paper_2608_00029_amd", "csrc"),
                    os.path.join(ROOT, "tests", "sched_check.cpp"), "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "bad=0" in out.stdout
