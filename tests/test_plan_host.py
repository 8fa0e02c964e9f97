"""Host check of the launch planner (CPU, no GPU): tests/plan_check.cpp,
compiled with the system C++ compiler against the library's planner source,
builds prefill and decode plans for random batches, masks and shapes and
verifies from the plan image that it fits the workspace's bound and that
the GEMM tiles and decode segments cover each active (row, head / K-V head /
FFN slice / K chunk) exactly once and nothing inactive."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_planner_coverage_and_bounds(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "plan_check")
    cmd = [cxx, "-std=c++20", "-O2", f"-I{os.path.join(ROOT, 'include')}",
           os.path.join(ROOT, "tests", "plan_check.cpp"),
           os.path.join(ROOT, "paper_2607_20357_amd", "csrc", "plan.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "plan_check ok" in r.stdout
