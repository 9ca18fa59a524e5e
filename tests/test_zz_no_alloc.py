"""pat_reducescatter_noalloc (the entry point that allocates nothing) against
pat_reducescatter, through the C-ABI.

Bar: the same bits as the allocating entry point on the same inputs (both
reach the PAT association), which in turn are checked here against the CPU
oracle: float32 / bf16 bit-exact against the PAT order and within 1e-5 / 1e-2
of the fp64 sum.  Calls come in a row on one stream, the second with a smaller
operation than the first, then the first again on new buffers: each call must
find whatever the previous one left in the shared scratch array and still be
exact.  No call may create a plan or take device memory.
"""

import sys

import numpy as np
import pytest
import torch

import synth
from oracle import definitions as D
from oracle import native
from paper_2506_20252_amd import pat

pytestmark = pytest.mark.gpu

TORCH = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pat.lib()
    torch.cuda.set_device(0)
    yield
    pat.check(pat.pat_set_exec_mode("stream"))


def as_bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def oracle_check(got, n, count, dtype, dist, seed):
    exp = native.reducescatter(dtype, n, count, dist=dist, seed=seed)
    width = {"int32": np.uint32, "float32": np.uint32, "bfloat16": np.uint16}[dtype]
    assert (got.view(width) == exp["pat"].view(width)).all()
    if dtype != "int32":
        val = got.astype(np.float64) if dtype == "float32" else D.bf16_bits_to_f32(got).astype(np.float64)
        tol = 1e-5 if dtype == "float32" else 1e-2
        assert (np.abs(val - exp["sum"]) <= tol * exp["abs"]).all()


def test_noalloc_matches_the_allocating_entry_point():
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    # (N, count, dtype, distribution, seed): the small-size regime (N = 1000,
    # 256 B chunks, about 122 MiB of slots), then a smaller bf16 operation with
    # an odd count (relaxed vectors, float32 root accumulators), then the first
    # shape again on new buffers and another mode setting (which the entry
    # point ignores: it always launches per-step kernels).
    cases = [(1000, 64, "float32", "f32_pm1", 0x5041544, "stream"),
             (24, 1001, "bfloat16", "bf16_normal", 0x2401, "stream"),
             (1000, 64, "float32", "f32_pm1", 0x5041599, "graph"),
             (7, 4096, "int32", "int32_pm2p20", 0x77, "persistent")]
    for k, (n, count, dtype, dist, seed, mode) in enumerate(cases):
        log(f"[gpu] noalloc call {k}: reduce-scatter n={n} count={count} {dtype} seed={seed:#x} mode={mode}")
        send = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
        for x in range(n):
            synth.fill(send[x], dist, seed, x)
        ref = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
        out = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
        out.view(torch.uint8).fill_(0x7F)
        S, R, O = pat.pointer_array(list(send)), pat.pointer_array(list(ref)), pat.pointer_array(list(out))
        pat.check(pat.pat_set_exec_mode(mode))
        pat.check(pat.pat_reducescatter(S, R, count, dtype, pat.PAT_SUM, n, stream), "pat_reducescatter")
        torch.cuda.synchronize()
        st, plans0, bytes0 = pat.pat_cache_stats()
        free0, _ = torch.cuda.mem_get_info()
        pat.check(pat.pat_reducescatter_noalloc(S, O, count, dtype, pat.PAT_SUM, n, stream), "noalloc")
        torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info()
        st, plans1, bytes1 = pat.pat_cache_stats()
        assert (plans1, bytes1) == (plans0, bytes0), "the no-allocation call created a plan"
        if k > 0:  # the first call may still see the runtime load the code object that holds the array
            assert free1 == free0, f"device memory changed by {free0 - free1} bytes"
        got, want = as_bits(out), as_bits(ref)
        width = np.uint16 if dtype == "bfloat16" else np.uint32
        mism = int(np.count_nonzero(got.view(width) != want.view(width)))
        assert mism == 0, f"call {k}: {mism} elements differ from pat_reducescatter"
        oracle_check(got, n, count, dtype, dist, seed)
        # a repeated call with the same plan and buffers launches kernels only
        out.view(torch.uint8).fill_(0x7F)
        pat.check(pat.pat_reducescatter_noalloc(S, O, count, dtype, pat.PAT_SUM, n, stream), "noalloc again")
        torch.cuda.synchronize()
        assert (as_bits(out).view(width) == want.view(width)).all()
        del send, ref, out, S, R, O
    pat.check(pat.pat_set_exec_mode("stream"))


def test_noalloc_refuses_operations_beyond_its_array():
    """N = 64 with 1 MiB float32 chunks needs about 1.4 GiB of slots: refused
    with PAT_ERR_TOO_LARGE before anything is launched (the addresses are
    never dereferenced)."""
    n, count = 64, 262144
    st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, n, count, "float32")
    assert info["slot_bytes_total"] > pat.NOALLOC_SCRATCH_BYTES
    send = [0x10_0000_0000 + x * (n * count * 4) for x in range(n)]
    recv = [0x20_0000_0000 + x * (count * 4) for x in range(n)]
    stream = torch.cuda.current_stream()
    assert pat.pat_reducescatter_noalloc(send, recv, count, "float32", pat.PAT_SUM, n, stream) == \
        pat.PAT_ERR_TOO_LARGE
    assert pat.pat_status_string(pat.PAT_ERR_TOO_LARGE) == "PAT_ERR_TOO_LARGE"
    # and a call that fits still works afterwards
    dev = torch.device("cuda:0")
    n, count, seed = 6, 1024, 0x5041541
    send = torch.empty((n, n * count), dtype=torch.int32, device=dev)
    for x in range(n):
        synth.fill(send[x], "int32_pm2p20", seed, x)
    out = torch.empty((n, count), dtype=torch.int32, device=dev)
    pat.check(pat.pat_reducescatter_noalloc(list(send), list(out), count, "int32", pat.PAT_SUM, n, stream))
    torch.cuda.synchronize()
    oracle_check(as_bits(out), n, count, "int32", "int32_pm2p20", seed)
