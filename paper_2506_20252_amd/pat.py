"""ctypes binding of libpat.so: the C-ABI declared in include/pat.h, same names.

Argument marshalling only: every step of the collective runs in the HIP
kernels of the library.  Buffers may be given as integers (device addresses)
or as objects with ``data_ptr()`` (e.g. torch tensors); streams as integers
(hipStream_t) or objects with ``cuda_stream`` (torch streams); None is the
default stream.  Functions return the pat_status_t code, like the C calls;
``check()`` turns a non-zero code into an exception.

If the library is not built, loading it raises: there is no fallback.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpat.so")

PAT_OK = 0
PAT_ERR_INVALID_ARGUMENT = 1
PAT_ERR_UNSUPPORTED = 2
PAT_ERR_OUT_OF_MEMORY = 3
PAT_ERR_HIP = 4
PAT_ERR_TIMEOUT = 5
PAT_ERR_INTERNAL = 6
PAT_ERR_TOO_LARGE = 7

NOALLOC_SCRATCH_BYTES = 256 << 20  # PAT_NOALLOC_SCRATCH_BYTES

PAT_INT32 = 0
PAT_FLOAT32 = 1
PAT_BFLOAT16 = 2
DTYPES = {"int32": PAT_INT32, "float32": PAT_FLOAT32, "bfloat16": PAT_BFLOAT16}
ELEM_BYTES = {PAT_INT32: 4, PAT_FLOAT32: 4, PAT_BFLOAT16: 2}

PAT_SUM = 0

PAT_ALLGATHER = 0
PAT_REDUCESCATTER = 1

PAT_EXEC_PERSISTENT = 0
PAT_EXEC_GRAPH = 1
PAT_EXEC_STREAM = 2
PAT_EXEC_DATAFLOW = 3
MODES = {"persistent": PAT_EXEC_PERSISTENT, "graph": PAT_EXEC_GRAPH, "stream": PAT_EXEC_STREAM,
         "dataflow": PAT_EXEC_DATAFLOW}

PAT_LINEAR_FAR_FIRST = 0
PAT_LINEAR_CLOSE_FIRST = 1
ORDERS = {"far": PAT_LINEAR_FAR_FIRST, "close": PAT_LINEAR_CLOSE_FIRST}

PAT_FUSION_AUTO = 0
PAT_FUSION_OFF = 1
PAT_FUSION_ON = 2
FUSIONS = {"auto": PAT_FUSION_AUTO, "off": PAT_FUSION_OFF, "on": PAT_FUSION_ON}

PAT_AGGREGATION_POW2 = 0
PAT_AGGREGATION_BUDGET = 1
AGGREGATIONS = {"pow2": PAT_AGGREGATION_POW2, "budget": PAT_AGGREGATION_BUDGET}

# Every function include/pat.h declares.
EXPORTS = (
    "pat_allgather", "pat_reducescatter", "pat_reducescatter_noalloc", "pat_set_buffer_bytes", "pat_get_buffer_bytes",
    "pat_set_exec_mode", "pat_get_exec_mode", "pat_set_linear_order", "pat_get_linear_order",
    "pat_set_top_fusion", "pat_get_top_fusion", "pat_set_aggregation", "pat_get_aggregation",
    "pat_set_barrier_timeout_us", "pat_plan_info",
    "pat_plan_steps", "pat_trace_start", "pat_trace_read", "pat_step_clock", "pat_cache_stats",
    "pat_check_device_status", "pat_last_hip_error", "pat_status_string",
    "pat_finalize",
)


class pat_plan_info_t(ctypes.Structure):
    _fields_ = [
        ("nranks", ctypes.c_int), ("L", ctypes.c_int), ("t", ctypes.c_int), ("T", ctypes.c_int),
        ("steps", ctypes.c_int), ("pieces", ctypes.c_int), ("max_chunks_per_step", ctypes.c_int),
        ("vector_path", ctypes.c_int), ("count", ctypes.c_size_t), ("piece_elems", ctypes.c_size_t),
        ("slot_elem_bytes", ctypes.c_size_t), ("slot_dims", ctypes.c_int),
        ("slot_chunks_per_rank", ctypes.c_int), ("slot_bytes_per_rank", ctypes.c_size_t),
        ("slot_bytes_total", ctypes.c_size_t), ("alg_bytes", ctypes.c_double),
        ("bus_bytes_per_rank", ctypes.c_double), ("fused_steps", ctypes.c_int),
        ("launches_per_op", ctypes.c_int), ("streaming", ctypes.c_int), ("xcd_run", ctypes.c_int),
        ("list_schedule", ctypes.c_int),
    ]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class PatError(RuntimeError):
    def __init__(self, status, where=""):
        self.status = status
        super().__init__(f"{where}: {pat_status_string(status)}"
                         + (f" (hipError {pat_last_hip_error()})" if status == PAT_ERR_HIP else ""))


_lib = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "pat_allgather": ([_P, _P, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, _P], ctypes.c_int),
            "pat_reducescatter": ([_P, _P, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int, _P],
                                  ctypes.c_int),
            "pat_reducescatter_noalloc": ([_P, _P, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int, _P],
                                          ctypes.c_int),
            "pat_set_buffer_bytes": ([ctypes.c_size_t], ctypes.c_int),
            "pat_get_buffer_bytes": ([], ctypes.c_size_t),
            "pat_set_exec_mode": ([ctypes.c_int], ctypes.c_int),
            "pat_get_exec_mode": ([], ctypes.c_int),
            "pat_set_linear_order": ([ctypes.c_int], ctypes.c_int),
            "pat_get_linear_order": ([], ctypes.c_int),
            "pat_set_top_fusion": ([ctypes.c_int], ctypes.c_int),
            "pat_get_top_fusion": ([], ctypes.c_int),
            "pat_set_aggregation": ([ctypes.c_int], ctypes.c_int),
            "pat_get_aggregation": ([], ctypes.c_int),
            "pat_set_barrier_timeout_us": ([ctypes.c_uint32], ctypes.c_int),
            "pat_plan_info": ([ctypes.c_int, ctypes.c_int, ctypes.c_size_t, ctypes.c_int,
                               ctypes.POINTER(pat_plan_info_t)], ctypes.c_int),
            "pat_plan_steps": ([ctypes.c_int, ctypes.c_int, ctypes.c_size_t, ctypes.c_int, _I32P, _I32P,
                                ctypes.c_int, _I32P, _I32P, _I32P, _I32P, ctypes.c_int,
                                ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)], ctypes.c_int),
            "pat_trace_start": ([ctypes.c_int], ctypes.c_int),
            "pat_trace_read": ([ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double), _I32P, _I32P,
                                ctypes.c_int, ctypes.POINTER(ctypes.c_int)], ctypes.c_int),
            "pat_step_clock": ([ctypes.c_int, ctypes.c_int, ctypes.c_size_t, ctypes.c_int,
                                ctypes.POINTER(ctypes.c_uint64), ctypes.c_size_t, ctypes.POINTER(ctypes.c_int),
                                ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
            "pat_cache_stats": ([ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
            "pat_check_device_status": ([_P], ctypes.c_int),
            "pat_last_hip_error": ([], ctypes.c_int),
            "pat_status_string": ([ctypes.c_int], ctypes.c_char_p),
            "pat_finalize": ([], ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def check(status, where="pat"):
    if status != PAT_OK:
        raise PatError(status, where)
    return status


def _dtype(dtype):
    return DTYPES[dtype] if isinstance(dtype, str) else int(dtype)


def _addr(b):
    return int(b.data_ptr()) if hasattr(b, "data_ptr") else int(b)


def pointer_array(bufs):
    """A ctypes array of device addresses, to build once and pass on every call
    (the entry points accept it as is)."""
    if isinstance(bufs, ctypes.Array):
        return bufs
    vals = [_addr(b) for b in bufs]
    return (ctypes.c_void_p * max(len(vals), 1))(*vals)


_ptr_array = pointer_array


def _stream(stream):
    if stream is None:
        return None
    if hasattr(stream, "cuda_stream"):
        return int(stream.cuda_stream)
    return int(stream)


def pat_allgather(sendbufs, recvbufs, count, dtype, nranks, stream=None):
    return lib().pat_allgather(_ptr_array(sendbufs), _ptr_array(recvbufs), int(count), _dtype(dtype),
                               int(nranks), _stream(stream))


def pat_reducescatter(sendbufs, recvbufs, count, dtype, op, nranks, stream=None):
    return lib().pat_reducescatter(_ptr_array(sendbufs), _ptr_array(recvbufs), int(count), _dtype(dtype),
                                   int(op), int(nranks), _stream(stream))


def pat_reducescatter_noalloc(sendbufs, recvbufs, count, dtype, op, nranks, stream=None):
    return lib().pat_reducescatter_noalloc(_ptr_array(sendbufs), _ptr_array(recvbufs), int(count), _dtype(dtype),
                                           int(op), int(nranks), _stream(stream))


# ---------------------------------------------------------------------------
# Tensor-level convenience: the same two calls, with the rank count, count and
# dtype read from torch tensors.  Marshalling only; the checks below are the
# shapes and placement the C calls document (device memory, element-contiguous
# rows).  Building the pointer arrays costs O(N) Python
# per call: a caller in a hot loop builds them once with pointer_array() and
# calls pat_allgather / pat_reducescatter directly.
# ---------------------------------------------------------------------------

_TORCH_DTYPES = {"torch.int32": "int32", "torch.float32": "float32", "torch.bfloat16": "bfloat16"}


def _rows(t, what):
    """A 2-D tensor is one row per rank; a list or tuple is taken as is."""
    if isinstance(t, (list, tuple)):
        return list(t)
    if getattr(t, "dim", lambda: 0)() != 2:
        raise ValueError(f"{what}: a 2-D tensor (one row per rank) or a list of per-rank tensors")
    return list(t)


def _check_rows(rows, what):
    """Every row must be a contiguous device tensor, all on one GPU: the
    kernels take each row's address as `numel` consecutive elements.  Returns
    that device."""
    devices = set()
    for r in rows:
        if not hasattr(r, "is_cuda") or not r.is_cuda:
            raise ValueError(f"{what}: every row must be a GPU tensor (a host address would reach the kernels)")
        if not (r.is_contiguous() or (r.dim() == 1 and r.numel() <= 1)):
            raise ValueError(f"{what}: every row must be contiguous (its elements consecutive in memory)")
        devices.add(r.device)
    if len(devices) > 1:
        raise ValueError(f"{what}: all rows must be on one device, got {sorted(str(d) for d in devices)}")
    return next(iter(devices))


def _dtype_of(rows, what):
    names = {str(r.dtype) for r in rows}
    if len(names) != 1 or next(iter(names)) not in _TORCH_DTYPES:
        raise ValueError(f"{what}: one dtype of int32, float32 or bfloat16 for every rank, got {sorted(names)}")
    return _TORCH_DTYPES[next(iter(names))]


def _tensor_call_stream(device, stream):
    """The stream a tensor-level call runs on: the one given, else torch's
    current stream of the rows' device (so that the call is ordered after the
    work that produced its inputs, also inside ``torch.cuda.stream(...)``).
    The rows must be on the current device: the library plans per current
    device."""
    import torch
    if device != torch.device("cuda", torch.cuda.current_device()):
        raise ValueError(f"rows are on {device}, but the current device is cuda:{torch.cuda.current_device()}")
    return stream if stream is not None else torch.cuda.current_stream(device)


def allgather(send, recv, stream=None):
    """recv[r] = concatenation of send[0..N-1] for every rank r.  send: N rows
    of `count` elements; recv: N rows of N * count elements, same dtype, all
    on the current GPU with unit stride.  Runs on `stream`, by default torch's
    current stream.  Raises ValueError on bad rows, PatError on a failed call."""
    s_rows, r_rows = _rows(send, "send"), _rows(recv, "recv")
    n = len(s_rows)
    if n < 1 or len(r_rows) != n:
        raise ValueError("send and recv need one row per rank, as many of each")
    count = s_rows[0].numel()
    if any(r.numel() != count for r in s_rows) or any(r.numel() != n * count for r in r_rows):
        raise ValueError("send rows hold `count` elements, recv rows N * count")
    dtype = _dtype_of(s_rows + r_rows, "allgather")
    stream = _tensor_call_stream(_check_rows(s_rows + r_rows, "allgather"), stream)
    return check(pat_allgather(s_rows, r_rows, count, dtype, n, stream), "pat_allgather")


def reducescatter(send, recv, stream=None):
    """recv[R] = sum over x of send[x][R * count : (R + 1) * count].  send: N
    rows of N * count elements; recv: N rows of `count`, same dtype (bf16
    sums accumulate in float32), all on the current GPU with unit stride.
    Runs on `stream`, by default torch's current stream.  Raises ValueError on
    bad rows, PatError on a failed call."""
    s_rows, r_rows = _rows(send, "send"), _rows(recv, "recv")
    n = len(s_rows)
    if n < 1 or len(r_rows) != n:
        raise ValueError("send and recv need one row per rank, as many of each")
    count = r_rows[0].numel()
    if any(r.numel() != count for r in r_rows) or any(r.numel() != n * count for r in s_rows):
        raise ValueError("recv rows hold `count` elements, send rows N * count")
    dtype = _dtype_of(s_rows + r_rows, "reducescatter")
    stream = _tensor_call_stream(_check_rows(s_rows + r_rows, "reducescatter"), stream)
    return check(pat_reducescatter(s_rows, r_rows, count, dtype, PAT_SUM, n, stream), "pat_reducescatter")


def pat_set_buffer_bytes(nbytes):
    return lib().pat_set_buffer_bytes(int(nbytes))


def pat_get_buffer_bytes():
    return int(lib().pat_get_buffer_bytes())


def pat_set_exec_mode(mode):
    return lib().pat_set_exec_mode(MODES[mode] if isinstance(mode, str) else int(mode))


def pat_get_exec_mode():
    return int(lib().pat_get_exec_mode())


def pat_set_top_fusion(mode):
    return lib().pat_set_top_fusion(FUSIONS[mode] if isinstance(mode, str) else int(mode))


def pat_get_top_fusion():
    return int(lib().pat_get_top_fusion())


def pat_set_aggregation(mode):
    return lib().pat_set_aggregation(AGGREGATIONS[mode] if isinstance(mode, str) else int(mode))


def pat_get_aggregation():
    return int(lib().pat_get_aggregation())


def pat_set_linear_order(order):
    return lib().pat_set_linear_order(ORDERS[order] if isinstance(order, str) else int(order))


def pat_get_linear_order():
    return int(lib().pat_get_linear_order())


def pat_set_barrier_timeout_us(microseconds):
    return lib().pat_set_barrier_timeout_us(int(microseconds))


def pat_plan_info(coll, nranks, count, dtype):
    """Returns (status, dict)."""
    info = pat_plan_info_t()
    st = lib().pat_plan_info(int(coll), int(nranks), int(count), _dtype(dtype), ctypes.byref(info))
    return st, info.as_dict()


def pat_plan_steps(coll, nranks, count, dtype):
    """Returns (status, steps, entries): steps = [(d, k)], entries = [(p, a, b, c)]."""
    n = max(int(nranks), 1)
    d = (ctypes.c_int32 * n)()
    k = (ctypes.c_int32 * n)()
    pos, a, b, c = [(ctypes.c_int32 * n)() for _ in range(4)]
    ns, ne = ctypes.c_int(), ctypes.c_int()
    st = lib().pat_plan_steps(int(coll), int(nranks), int(count), _dtype(dtype), d, k, n, pos, a, b, c, n,
                              ctypes.byref(ns), ctypes.byref(ne))
    if st != PAT_OK:
        return st, [], []
    steps = [(d[i], k[i]) for i in range(ns.value)]
    entries = [(pos[j], a[j], b[j], c[j]) for j in range(ne.value)]
    return st, steps, entries


def pat_trace_start(max_launches):
    return lib().pat_trace_start(int(max_launches))


def pat_trace_read(max_launches):
    """Returns (status, launches): launches = [(ms, bytes, kind, step)] in launch order."""
    m = max(int(max_launches), 1)
    ms, by = (ctypes.c_float * m)(), (ctypes.c_double * m)()
    kind, step = (ctypes.c_int32 * m)(), (ctypes.c_int32 * m)()
    n = ctypes.c_int()
    st = lib().pat_trace_read(ms, by, kind, step, m, ctypes.byref(n))
    if st != PAT_OK:
        return st, []
    return st, [(ms[j], by[j], kind[j], step[j]) for j in range(n.value)]


def pat_step_clock(coll, nranks, count, dtype):
    """Returns (status, stamps, ticks_per_us): stamps is a (workgroups,
    steps + 1) numpy array of device wall-clock ticks of the plan's last fused
    launch (PAT_STEP_CLOCK=1), or None."""
    import numpy as np
    wgs, per, tpu = ctypes.c_int(), ctypes.c_int(), ctypes.c_double()
    st = lib().pat_step_clock(int(coll), int(nranks), int(count), _dtype(dtype), None, 0, ctypes.byref(wgs),
                              ctypes.byref(per), ctypes.byref(tpu))
    if wgs.value == 0:
        return st, None, 0.0
    out = np.zeros((wgs.value, per.value), dtype=np.uint64)
    st = lib().pat_step_clock(int(coll), int(nranks), int(count), _dtype(dtype),
                              out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), out.size, ctypes.byref(wgs),
                              ctypes.byref(per), ctypes.byref(tpu))
    return st, (out if st == PAT_OK else None), tpu.value


def pat_cache_stats():
    """Returns (status, number of cached plans, device bytes they hold)."""
    n, b = ctypes.c_int(), ctypes.c_size_t()
    st = lib().pat_cache_stats(ctypes.byref(n), ctypes.byref(b))
    return st, n.value, b.value


def pat_check_device_status(stream=None):
    return lib().pat_check_device_status(_stream(stream))


def pat_last_hip_error():
    return int(lib().pat_last_hip_error())


def pat_status_string(status):
    return lib().pat_status_string(int(status)).decode()


def pat_finalize():
    return lib().pat_finalize()
