"""ctypes binding of the threaded C++ oracle (oracle/liboracle.so).

Test infrastructure only (see the package docstring).  ``reducescatter``
returns the reduce-scatter's expected results for a range of destination
chunks: the PAT association (the reversed-tree closed form, section
"Conversion to reduce-scatter operations"), the plain fp64 sum over ranks and
the fp64 sum of absolute values (section "All-gather and reduce-scatter
algorithms").  ``allgather`` returns the all-gather's result rows for a range
of receivers: the concatenation of every rank's send buffer (the same
section).  Inputs are either arrays or regenerated from the seeded generator
of ``synth`` (the same values the device fill writes), so that operations far
larger than host memory can be checked, or timed, block by block.
"""

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

_DTYPES = {"int32": (0, np.int32), "float32": (1, np.float32), "bfloat16": (2, np.uint16)}
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.oracle_reducescatter.argtypes = [P, ctypes.c_int, ctypes.c_uint64, ctypes.c_int64, ctypes.c_uint64, P,
                                           ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           P, P, P, ctypes.c_int]
        L.oracle_reducescatter.restype = ctypes.c_int
        L.oracle_allgather.argtypes = [P, ctypes.c_int, ctypes.c_uint64, ctypes.c_int64, ctypes.c_uint64, P,
                                       ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int, P,
                                       ctypes.c_int]
        L.oracle_allgather.restype = ctypes.c_int
        L.oracle_threads.argtypes = []
        L.oracle_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def threads():
    """Host threads the oracle uses by default (the CPUs this process may run on)."""
    return int(lib().oracle_threads())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def reducescatter(dtype, nranks, count, inputs=None, dist=None, seed=0, r0=0, r1=None,
                  want=("pat", "sum", "abs"), nthreads=0):
    """Expected reduce-scatter results for destination chunks [r0, r1).

    inputs: (N, N, count) array (bf16 as uint16 bit patterns), or None to
    regenerate rank x's send buffer from ``synth`` distribution `dist` and
    `seed`.  Returns a dict with the requested arrays, each (r1 - r0, count):
    "pat" in the input dtype (the PAT association), "sum" and "abs" in fp64,
    and "threads", the worker count used."""
    import synth

    code, np_dtype = _DTYPES[dtype]
    r1 = nranks if r1 is None else r1
    rows = r1 - r0
    out = {}
    if "pat" in want:
        out["pat"] = np.empty((rows, count), dtype=np_dtype)
    for k in ("sum", "abs"):
        if k in want:
            out[k] = np.empty((rows, count), dtype=np.float64)
    kind, lo, span, table = 0, 0, 0, None
    if inputs is not None:
        inputs = np.ascontiguousarray(inputs)
        if inputs.shape != (nranks, nranks, count) or inputs.dtype != np_dtype:
            raise ValueError(f"inputs: ({nranks}, {nranks}, {count}) {np.dtype(np_dtype).name} expected")
    else:
        spec = synth.DISTS[dist]
        kind, lo, span = spec["kind"], spec["lo"], spec["span"]
        if kind >= 2:
            table = np.ascontiguousarray(synth.normal_table(dist))
    used = lib().oracle_reducescatter(_ptr(inputs), kind, seed & 0xFFFFFFFFFFFFFFFF, lo, span, _ptr(table),
                                      nranks, count, code, r0, r1, _ptr(out.get("pat")), _ptr(out.get("sum")),
                                      _ptr(out.get("abs")), nthreads)
    if used < 0:
        raise ValueError("oracle_reducescatter: invalid arguments")
    out["threads"] = used
    return out


def allgather(dtype, nranks, count, inputs=None, dist=None, seed=0, r0=0, r1=None, nthreads=0, out=None):
    """All-gather result rows of receivers [r0, r1): (r1 - r0, N * count) in
    the input dtype (bf16 as uint16 bit patterns), each the concatenation of
    the N send buffers.  inputs: (N, count) array, or None to regenerate rank
    x's send buffer from ``synth`` distribution `dist` and `seed`.  `out` may
    supply the result array (reused across blocks).  Returns (rows, threads)."""
    import synth

    code, np_dtype = _DTYPES[dtype]
    r1 = nranks if r1 is None else r1
    shape = (r1 - r0, nranks * count)
    if out is None:
        out = np.empty(shape, dtype=np_dtype)
    elif out.shape != shape or out.dtype != np_dtype or not out.flags["C_CONTIGUOUS"]:
        raise ValueError(f"out: contiguous {shape} {np.dtype(np_dtype).name} expected")
    kind, lo, span, table = 0, 0, 0, None
    if inputs is not None:
        inputs = np.ascontiguousarray(inputs)
        if inputs.shape != (nranks, count) or inputs.dtype != np_dtype:
            raise ValueError(f"inputs: ({nranks}, {count}) {np.dtype(np_dtype).name} expected")
    else:
        spec = synth.DISTS[dist]
        kind, lo, span = spec["kind"], spec["lo"], spec["span"]
        if kind >= 2:
            table = np.ascontiguousarray(synth.normal_table(dist))
    used = lib().oracle_allgather(_ptr(inputs), kind, seed & 0xFFFFFFFFFFFFFFFF, lo, span, _ptr(table), nranks,
                                  count, code, r0, r1, _ptr(out), nthreads)
    if used < 0:
        raise ValueError("oracle_allgather: invalid arguments")
    return out, used
