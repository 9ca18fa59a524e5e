"""C-ABI boundary checks that need no GPU: the library loads, exports every
function include/pat.h declares, and rejects bad arguments before touching
the device."""

import ctypes
import os
import re

import pytest

from paper_2506_20252_amd import pat

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "pat.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pat_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 13
    lib = ctypes.CDLL(pat.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(pat.EXPORTS) == names


def test_status_strings():
    assert pat.pat_status_string(pat.PAT_OK) == "PAT_OK"
    assert pat.pat_status_string(pat.PAT_ERR_TIMEOUT) == "PAT_ERR_TIMEOUT"
    assert pat.pat_status_string(99) == "PAT_ERR_UNKNOWN"


def fake(base, n, stride):
    return [base + i * stride for i in range(n)]


def test_argument_errors_before_any_device_call():
    ok_send = fake(0x100000, 4, 0x10000)
    ok_recv = fake(0x900000, 4, 0x10000)
    # count == 0 is a no-op
    assert pat.pat_allgather(ok_send, ok_recv, 0, "float32", 4) == pat.PAT_OK
    assert pat.pat_reducescatter(ok_send, ok_recv, 0, "int32", pat.PAT_SUM, 4) == pat.PAT_OK
    # rank count
    assert pat.pat_allgather(ok_send, ok_recv, 16, "float32", 0) == pat.PAT_ERR_INVALID_ARGUMENT
    assert pat.pat_allgather(ok_send, ok_recv, 16, "float32", -3) == pat.PAT_ERR_INVALID_ARGUMENT
    # dtype / op
    assert pat.pat_allgather(ok_send, ok_recv, 16, 7, 4) == pat.PAT_ERR_UNSUPPORTED
    assert pat.pat_reducescatter(ok_send, ok_recv, 16, "float32", 3, 4) == pat.PAT_ERR_UNSUPPORTED
    # null buffer
    assert pat.pat_allgather(ok_send[:3] + [0], ok_recv, 16, "float32", 4) == pat.PAT_ERR_INVALID_ARGUMENT
    # element misalignment
    bad = list(ok_send)
    bad[2] += 2
    assert pat.pat_allgather(bad, ok_recv, 16, "float32", 4) == pat.PAT_ERR_INVALID_ARGUMENT
    # receive buffers overlapping each other (all-gather: 4 * 16 * 4 bytes each)
    assert pat.pat_allgather(ok_send, fake(0x900000, 4, 64), 16, "float32", 4) == pat.PAT_ERR_INVALID_ARGUMENT
    # a send buffer inside another rank's receive buffer
    assert pat.pat_allgather([0x900000 + 64] + ok_send[1:], ok_recv, 16, "float32", 4) == \
        pat.PAT_ERR_INVALID_ARGUMENT
    # in place, but at the wrong chunk
    inplace_wrong = [ok_recv[r] + ((r + 1) % 4) * 64 for r in range(4)]
    assert pat.pat_allgather(inplace_wrong, ok_recv, 16, "float32", 4) == pat.PAT_ERR_INVALID_ARGUMENT
    # reduce-scatter: receive buffer inside the own send buffer but not at chunk r
    rs_wrong = [ok_send[r] + ((r + 1) % 4) * 64 for r in range(4)]
    assert pat.pat_reducescatter(ok_send, rs_wrong, 16, "float32", pat.PAT_SUM, 4) == \
        pat.PAT_ERR_INVALID_ARGUMENT


def test_settings_roundtrip():
    assert pat.pat_set_exec_mode(5) == pat.PAT_ERR_INVALID_ARGUMENT
    old = pat.pat_get_exec_mode()
    assert pat.pat_set_exec_mode("graph") == pat.PAT_OK and pat.pat_get_exec_mode() == pat.PAT_EXEC_GRAPH
    assert pat.pat_set_exec_mode(old) == pat.PAT_OK
    assert pat.pat_set_buffer_bytes(1 << 20) == pat.PAT_OK and pat.pat_get_buffer_bytes() == 1 << 20
    assert pat.pat_set_buffer_bytes(0) == pat.PAT_OK and pat.pat_get_buffer_bytes() == 8 << 20
    assert pat.pat_finalize() == pat.PAT_OK  # nothing allocated: no device call
    assert pat.pat_cache_stats() == (pat.PAT_OK, 0, 0)


def test_plan_info_workloads():
    mib = 1 << 20
    cases = [
        # (coll, N, count, dtype, steps, T, pieces)
        (pat.PAT_REDUCESCATTER, 6, 1024, "int32", 3, 4, 1),
        (pat.PAT_ALLGATHER, 24, 32768, "bfloat16", 5, 16, 1),
        (pat.PAT_REDUCESCATTER, 64, 262144, "float32", 10, 8, 1),
        (pat.PAT_ALLGATHER, 1000, 64, "float32", 10, 512, 1),
        (pat.PAT_REDUCESCATTER, 1000, 64, "float32", 10, 512, 1),
        (pat.PAT_REDUCESCATTER, 128, 2 * mib, "bfloat16", 127, 1, 1),
    ]
    for coll, n, count, dt, steps, T, pieces in cases:
        st, info = pat.pat_plan_info(coll, n, count, dt)
        assert st == pat.PAT_OK
        assert (info["steps"], info["T"], info["pieces"]) == (steps, T, pieces), (n, info)
        assert info["slot_dims"] <= info["L"]
    # bf16 reduce-scatter carries float32 partials
    st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, 128, 2 * mib, "bfloat16")
    assert info["slot_elem_bytes"] == 4
    assert info["alg_bytes"] == pytest.approx(316.5 * 2**30, rel=1e-3)
    # a chunk larger than the budget: T = 1, pieces
    pat.pat_set_buffer_bytes(1 << 20)
    try:
        st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, 64, 262144 * 3, "float32")
        assert info["T"] == 1 and info["pieces"] == 3 and info["steps"] == 63
        # logarithmic buffers, independent of size: same slot entries per rank at any count
        sizes = {pat.pat_plan_info(pat.PAT_ALLGATHER, 37, c, "float32")[1]["slot_chunks_per_rank"]
                 for c in (1 << 18, 1 << 19, 1 << 21)}
        assert len(sizes) == 1
    finally:
        pat.pat_set_buffer_bytes(0)


def test_ceiling_probe_library_exports_and_checks_arguments():
    """The benchmark's streaming-ceiling probes (not part of the collectives)
    load, export their entry points, and refuse null or misaligned buffers and
    sizes that are not whole 16-byte vectors before any launch."""
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2506_20252_amd", "libpatceiling.so"))
    invalid = 1  # hipErrorInvalidValue
    for name, nbuf in (("pat_ceiling_copy", 2), ("pat_ceiling_copy2", 3), ("pat_ceiling_add", 3),
                       ("pat_ceiling_read", 2)):
        fn = getattr(lib, name)
        fn.argtypes = [ctypes.c_void_p] * nbuf + [ctypes.c_size_t, ctypes.c_void_p]
        fn.restype = ctypes.c_int
        good = [0x100000 * (i + 1) for i in range(nbuf)]
        assert fn(*([None] + good[1:]), 4096, None) == invalid, name
        assert fn(*(good[:-1] + [good[-1] + 8]), 4096, None) == invalid, name
        assert fn(*good, 4100, None) == invalid, name
    fn = lib.pat_ceiling_write
    fn.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint32, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    assert fn(None, 4096, 0, None) == invalid
    assert fn(0x100008, 4096, 0, None) == invalid
    assert fn(0x100000, 4100, 0, None) == invalid


def test_tensor_wrappers_check_shapes_and_dtypes_before_any_call():
    """The tensor-level allgather / reducescatter read N, count and dtype from
    the tensors and refuse inconsistent ones with ValueError before calling
    the library (host tensors here: no call may reach a device)."""
    import torch

    bad = [
        (pat.allgather, torch.zeros(4, 3), torch.zeros(4, 11)),                 # recv rows not N * count
        (pat.allgather, torch.zeros(4, 3), torch.zeros(3, 12)),                 # rank counts differ
        (pat.allgather, torch.zeros(4, 3, dtype=torch.float64), torch.zeros(4, 12, dtype=torch.float64)),
        (pat.allgather, torch.zeros(4, 3), torch.zeros(4, 12, dtype=torch.bfloat16)),  # mixed dtypes
        (pat.allgather, torch.zeros(12), torch.zeros(48)),                      # 1-D: rows unknown
        (pat.reducescatter, torch.zeros(4, 12), torch.zeros(4, 4)),             # send rows not N * count
        (pat.reducescatter, [torch.zeros(12)] * 4, [torch.zeros(3)] * 3),
        (pat.reducescatter, torch.zeros(0, 0), torch.zeros(0, 0)),              # no ranks
    ]
    for fn, send, recv in bad:
        with pytest.raises(ValueError):
            fn(send, recv)


class _FakeRow:
    """Just enough of a tensor for the binding's row checks (no GPU needed)."""

    def __init__(self, cuda=True, contiguous=True, device="cuda:0", dtype="torch.float32", numel=8):
        import torch
        self.is_cuda = cuda
        self._contiguous = contiguous
        self.device = torch.device(device)
        self.dtype = dtype
        self._numel = numel

    def is_contiguous(self):
        return self._contiguous

    def dim(self):
        return 1

    def numel(self):
        return self._numel

    def data_ptr(self):
        raise AssertionError("a rejected row must never reach the C call")


def test_tensor_wrappers_reject_host_tensors():
    """Host tensors never reach the kernels as addresses: the wrappers raise."""
    import torch
    send = torch.zeros((4, 8), dtype=torch.float32)
    with pytest.raises(ValueError, match="GPU tensor"):
        pat.allgather(send, torch.zeros((4, 32), dtype=torch.float32))
    with pytest.raises(ValueError, match="GPU tensor"):
        pat.reducescatter(torch.zeros((4, 32), dtype=torch.float32), send)


def test_tensor_wrappers_reject_strided_and_mixed_device_rows():
    rows = [_FakeRow() for _ in range(3)]
    assert str(pat._check_rows(rows, "x")) == "cuda:0"
    with pytest.raises(ValueError, match="contiguous"):
        pat._check_rows(rows + [_FakeRow(contiguous=False)], "x")
    with pytest.raises(ValueError, match="one device"):
        pat._check_rows(rows + [_FakeRow(device="cuda:1")], "x")
    with pytest.raises(ValueError, match="GPU tensor"):
        pat._check_rows(rows + [_FakeRow(cuda=False)], "x")
