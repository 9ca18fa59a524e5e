"""Compile the HIP libraries in place for gfx950 (hipcc cross-compiles; no GPU needed).

* paper_2506_20252_amd/libpat.so -- the PAT collectives (C-ABI of include/pat.h)
* synth/libpatsynth.so           -- the seeded input filler used by tests and the benchmark
* paper_2506_20252_amd/libpatceiling.so -- streaming-ceiling probes (a copy, a copy into two buffers,
                                          a 2-read/1-write add) that the benchmark reports beside
                                          the collectives
"""

import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2506_20252_amd")
CSRC = os.path.join(PKG, "csrc")

# -packed-fp32-ops: keep hipcc from emitting packed fp32 arithmetic.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

TARGETS = [
    (os.path.join(PKG, "libpat.so"),
     [os.path.join(CSRC, f) for f in ("plan.cpp", "api.cpp", "kernels.hip", "noalloc.hip")]),
    (os.path.join(ROOT, "synth", "libpatsynth.so"), [os.path.join(ROOT, "synth", "synth.hip")]),
    (os.path.join(PKG, "libpatceiling.so"), [os.path.join(CSRC, "ceiling.hip")]),
]


def hipcc():
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def build(verbose=False):
    for out, srcs in TARGETS:
        tmp = out + ".tmp"
        cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"build failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
        os.replace(tmp, out)
        if verbose:
            print("built", out)


if __name__ == "__main__":
    build(verbose=True)
