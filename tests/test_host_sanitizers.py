"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (g++, host
code only): the plan code driven over many plans by tests/host/plan_check.cpp,
the C-ABI layer against launch stubs driven by tests/host/api_check.cpp, and
the threaded C++ oracle (also under ThreadSanitizer) driven by
tests/host/oracle_check.cpp."""

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


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists("/opt/rocm/lib/libamdhip64.so"),
                    reason="no g++ or no HIP runtime library")
def test_abi_host_paths_under_asan_ubsan(tmp_path):
    """The C-ABI layer (api.cpp) built with g++ against do-nothing launch stubs
    (tests/host/api_stubs.cpp: no kernel ever runs), driven by
    tests/host/api_check.cpp: plan introspection over every shape and setting,
    and the argument checks with the remembered pointer set."""
    exe = tmp_path / "api_check"
    csrc = os.path.join(ROOT, "paper_2506_20252_amd", "csrc")
    host = os.path.join(ROOT, "tests", "host")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", csrc,
           os.path.join(csrc, "api.cpp"), os.path.join(csrc, "plan.cpp"),
           os.path.join(host, "api_stubs.cpp"), os.path.join(host, "api_check.cpp"),
           "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    # the HIP runtime's own start-up allocations are not ours to leak-check
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600,
                         env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert res.returncode == 0, (res.stdout[-1000:], res.stderr[-2000:])
    assert "plans checked, 0 failures" in res.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="no g++")
@pytest.mark.parametrize("sanitizer", ["address,undefined", "thread"])
def test_threaded_oracle_under_sanitizers(tmp_path, sanitizer):
    """The threaded C++ oracle (reduce-scatter and all-gather) driven by
    tests/host/oracle_check.cpp over every generator kind and dtype, ranks
    1 .. 100, empty and ragged counts, ranges and thread counts, under
    AddressSanitizer + UndefinedBehaviorSanitizer and under ThreadSanitizer."""
    exe = tmp_path / "oracle_check"
    oracle = os.path.join(ROOT, "oracle")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-pthread", f"-fsanitize={sanitizer}", "-fno-sanitize-recover=all",
           "-ffp-contract=off", "-I", ROOT, os.path.join(oracle, "rs_oracle.cpp"), os.path.join(oracle, "ag_oracle.cpp"),
           os.path.join(ROOT, "tests", "host", "oracle_check.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, (res.stdout[-1000:], res.stderr[-3000:])
    assert "oracle cases checked, 0 failures" in res.stdout
