"""Compile the threaded C++ oracle (oracle/liboracle.so) with g++.

Test infrastructure: the library is loaded only by tests/, __graft_entry__.smoke()
and the cpu_baseline leg of bench.py.  Plain C++17 and std::thread; no HIP.
-ffp-contract=off keeps every float32 add a single rounding (no fused
multiply-adds, no fast-math).
"""

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "liboracle.so")
FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", "-pthread", "-ffp-contract=off", "-fno-fast-math"]


def build(verbose=False):
    tmp = LIB_PATH + ".tmp"
    cmd = ["g++", *FLAGS, "-I", ROOT, os.path.join(HERE, "rs_oracle.cpp"), os.path.join(HERE, "ag_oracle.cpp"),
           "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"oracle build failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)


if __name__ == "__main__":
    build(verbose=True)
