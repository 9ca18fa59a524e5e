import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD Instinct GPU (gfx950) and the built HIP library")


def read_golden(name):
    """Parse a tests/golden fixture: '# ...' comments, 'key: values' lines."""
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, val = line.partition(":")
            out[key.strip()] = val.split()
    return out


def pytest_sessionstart(session):
    """Build the C++ oracle if it is missing or older than its source (g++,
    about a second; the HIP libraries are built by __graft_entry__.build())."""
    lib = os.path.join(ROOT, "oracle", "liboracle.so")
    srcs = [os.path.join(ROOT, "oracle", "rs_oracle.cpp"), os.path.join(ROOT, "synth", "synth_host.hpp")]
    if not os.path.exists(lib) or any(os.path.getmtime(s) > os.path.getmtime(lib) for s in srcs):
        from oracle import build as oracle_build
        oracle_build.build()
