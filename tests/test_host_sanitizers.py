"""The host plan code under AddressSanitizer and UndefinedBehaviorSanitizer
(g++, host code only; no HIP), driven over many plans by tests/host/plan_check.cpp."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="no g++")
def test_plan_code_under_asan_ubsan(tmp_path):
    exe = tmp_path / "plan_check"
    csrc = os.path.join(ROOT, "paper_2506_20252_amd", "csrc")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", csrc, os.path.join(csrc, "plan.cpp"), os.path.join(ROOT, "tests", "host", "plan_check.cpp"),
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert res.returncode == 0, res.stderr[-2000:]
    assert "plans checked" in res.stdout
