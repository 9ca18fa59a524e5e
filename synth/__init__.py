"""Seeded synthetic inputs: a device filler and its exact host twin.

This module serves both the HIP path's tests/benchmark and the CPU oracle's
checks.  It contains none of the collective's arithmetic: it maps
(seed, counter) to values with SplitMix64 (Steele, Lea, Flood, OOPSLA 2014),
identically in ``synth.hip`` (device) and in ``splitmix64_at`` below (host),
so the host can regenerate any element of a buffer the device filled.

Buffer convention: element i of rank x's send buffer uses counter
``(x << 36) + i``.

Distributions (one per workload family):

* ``int32_pm2p20``  -- int32 uniform on [-2^20, 2^20] (both ends included)
* ``f32_pm1``       -- float32 uniform on [-1, 1) in steps of 2^-23
* ``f32_normal``    -- float32 N(0, 1) by inverse-CDF table: 65536 equiprobable
  cells, value Phi^-1((k + 1/2) / 65536) rounded to float32, k = top 16 bits
* ``bf16_normal``   -- the same table rounded once more to bfloat16 (bit patterns)
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpatsynth.so")

GAMMA = 0x9E3779B97F4A7C15
M1 = 0xBF58476D1CE4E5B9
M2 = 0x94D049BB133111EB

DISTS = {
    "int32_pm2p20": dict(kind=0, np_dtype=np.int32, lo=-(1 << 20), span=(1 << 21) + 1),
    "f32_pm1": dict(kind=1, np_dtype=np.float32, lo=0, span=0),
    "f32_normal": dict(kind=3, np_dtype=np.float32, lo=0, span=0),
    "bf16_normal": dict(kind=2, np_dtype=np.uint16, lo=0, span=0),
}

RANK_SHIFT = 36


def counter_base(rank: int) -> int:
    return int(rank) << RANK_SHIFT


def splitmix64_at(seed: int, n: np.ndarray) -> np.ndarray:
    """Value n of the SplitMix64 stream seeded with `seed` (uint64 arithmetic)."""
    n = np.asarray(n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + (n + np.uint64(1)) * np.uint64(GAMMA)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(M2)
        return z ^ (z >> np.uint64(31))


_TABLES = {}


def normal_table(dist: str) -> np.ndarray:
    """65536-entry inverse-CDF table (float32 values, or bf16 bit patterns)."""
    if dist not in _TABLES:
        from scipy.special import ndtri
        k = np.arange(65536, dtype=np.float64)
        f32 = ndtri((k + 0.5) / 65536.0).astype(np.float32)
        if dist == "f32_normal":
            _TABLES[dist] = f32
        elif dist == "bf16_normal":
            import torch
            _TABLES[dist] = torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        else:
            raise ValueError(dist)
    return _TABLES[dist]


def host_values(dist: str, seed: int, rank: int, idx) -> np.ndarray:
    """Values of elements `idx` of rank `rank`'s buffer (host twin of the fill)."""
    spec = DISTS[dist]
    idx = np.asarray(idx, dtype=np.uint64)
    h = splitmix64_at(seed, np.uint64(counter_base(rank)) + idx)
    kind = spec["kind"]
    if kind == 0:
        off = ((h >> np.uint64(32)) * np.uint64(spec["span"])) >> np.uint64(32)
        return (off.astype(np.int64) + spec["lo"]).astype(np.int32)
    if kind == 1:
        k = (h >> np.uint64(40)).astype(np.int64) - (1 << 23)
        return k.astype(np.float32) * np.float32(2.0 ** -23)
    return normal_table(dist)[(h >> np.uint64(48)).astype(np.int64)]


def host_buffer(dist: str, seed: int, rank: int, n: int) -> np.ndarray:
    return host_values(dist, seed, rank, np.arange(n, dtype=np.uint64))


# ---------------------------------------------------------------------------
# Device fill (needs the built libpatsynth.so and a GPU)
# ---------------------------------------------------------------------------

_lib = None
_dev_tables = {}


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        lib.synth_fill.restype = ctypes.c_int
        lib.synth_fill.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                   ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p,
                                   ctypes.c_void_p]
        _lib = lib
    return _lib


def _device_table(dist: str, device):
    import torch
    key = (dist, str(device))
    if key not in _dev_tables:
        tab = normal_table(dist)
        _dev_tables[key] = torch.from_numpy(tab.view(np.int16 if tab.dtype == np.uint16 else np.int32).copy()).to(device)
    return _dev_tables[key]


def fill(tensor, dist: str, seed: int, rank: int, offset: int = 0, stream=None):
    """Fill a contiguous CUDA tensor as elements [offset, offset + numel) of
    rank `rank`'s buffer."""
    import torch
    spec = DISTS[dist]
    assert tensor.is_contiguous() and tensor.is_cuda
    table = 0
    if spec["kind"] >= 2:
        table = _device_table(dist, tensor.device).data_ptr()
    if stream is None:
        stream = torch.cuda.current_stream(tensor.device).cuda_stream
    rc = _load().synth_fill(tensor.data_ptr(), tensor.numel(), seed & 0xFFFFFFFFFFFFFFFF,
                            counter_base(rank) + offset, spec["kind"], spec["lo"], spec["span"],
                            table, stream)
    if rc != 0:
        raise RuntimeError(f"synth_fill failed with hipError {rc}")
