"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle.

Bars:
* all-gather: bit-exact (a byte copy);
* reduce-scatter int32: bit-exact (wrapping sum);
* reduce-scatter float32: bit-exact against the oracle executing the PAT
  steps (same association), and |got - sum| <= 1e-5 * sum|v| against the fp64
  plain sum;
* reduce-scatter bf16 (float32 partials): bit-exact against the oracle's PAT
  order, and within 1e-2 * sum|v| of the fp64 plain sum.

Inputs come from the seeded generator (device fill, host twin); the large
workloads are checked on sampled element positions the oracle computes one by
one (every element position is an independent reduction).
"""

import os
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import definitions as D
from oracle import native
from oracle import pat as opat
from paper_2506_20252_amd import pat

pytestmark = pytest.mark.gpu

TORCH = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}
DIST = {"int32": "int32_pm2p20", "float32": "f32_normal", "bfloat16": "bf16_normal"}
MIB = 1 << 20


def log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pat.lib()
    torch.cuda.set_device(0)
    os.environ["PAT_POISON_SLOTS"] = "1"  # slots start as 0xFF.. (NaN for floats)
    pat.check(pat.pat_finalize())
    yield
    pat.check(pat.pat_finalize())
    os.environ.pop("PAT_POISON_SLOTS", None)
    torch.cuda.empty_cache()


def as_bits(t):
    """Device tensor -> numpy with the oracle's conventions (bf16 as uint16)."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def fill_ranks(buf, dist, seed):
    for x in range(buf.shape[0]):
        synth.fill(buf[x], dist, seed, x)


def host_rs_inputs(n, count, dist, seed, sample=None):
    """(N, N, m): rank x's contribution to chunk R at the sampled positions."""
    if sample is None:
        return np.stack([synth.host_buffer(dist, seed, x, n * count) for x in range(n)]).reshape(n, n, count)
    idx = (np.arange(n, dtype=np.uint64)[:, None] * np.uint64(count) + sample.astype(np.uint64)[None, :])
    return np.stack([synth.host_values(dist, seed, x, idx.ravel()).reshape(n, len(sample)) for x in range(n)])


def check_rs(got, host_in, dtype, budget_t, order="far"):
    """got: (N, m) from the device; host_in: (N, N, m)."""
    if dtype == "int32":
        ref = D.reducescatter_sum(host_in, "int32")
        np.testing.assert_array_equal(got, ref)
        return
    pat_ref, _ = opat.reducescatter(host_in, budget_t, dtype, order)
    width = np.uint32 if dtype == "float32" else np.uint16
    mism = np.count_nonzero(got.view(width) != pat_ref.view(width))
    assert mism == 0, f"{mism} elements differ from the PAT-order oracle"
    exact = D.reducescatter_sum(host_in, dtype)
    scale = D.reducescatter_abs_sum(host_in, dtype)
    val = got.astype(np.float64) if dtype == "float32" else D.bf16_bits_to_f32(got).astype(np.float64)
    tol = 1e-5 if dtype == "float32" else 1e-2
    assert (np.abs(val - exact) <= tol * scale).all()


def oracle_t(coll, n, count, dtype):
    slot = 4 if (coll == pat.PAT_REDUCESCATTER or dtype != "bfloat16") else 2
    return opat.aggregation_level(n, count * slot, pat.pat_get_buffer_bytes())


def run_rs(n, count, dtype, seed, mode="persistent", inplace=False, sample=None, dist=None):
    log(f"[gpu] reduce-scatter n={n} count={count} dtype={dtype} seed={seed:#x} mode={mode} inplace={inplace}")
    dev = torch.device("cuda:0")
    send = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
    fill_ranks(send, dist or DIST[dtype], seed)
    if inplace:
        recvs = [send[r, r * count:(r + 1) * count] for r in range(n)]
    else:
        recv = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
        recv.view(torch.uint8).fill_(0x7F)
        recvs = list(recv)
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    pat.check(pat.pat_reducescatter(list(send), recvs, count, dtype, pat.PAT_SUM, n, stream), "rs")
    pat.check(pat.pat_check_device_status(stream), "status")
    out = torch.stack(recvs)
    if sample is not None:
        out = out[:, torch.as_tensor(sample, device=dev)]
    got = as_bits(out)
    del send, recvs, out
    return got


def run_ag(n, count, dtype, seed, mode="persistent", inplace=False, dist=None):
    log(f"[gpu] all-gather n={n} count={count} dtype={dtype} seed={seed:#x} mode={mode} inplace={inplace}")
    dist = dist or DIST[dtype]
    dev = torch.device("cuda:0")
    recv = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
    recv.view(torch.uint8).fill_(0xA5)
    if inplace:
        sends = [recv[r, r * count:(r + 1) * count] for r in range(n)]
        for r in range(n):
            synth.fill(sends[r], dist, seed, r)
    else:
        send = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
        fill_ranks(send, dist, seed)
        sends = list(send)
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    pat.check(pat.pat_allgather(sends, list(recv), count, dtype, n, stream), "ag")
    pat.check(pat.pat_check_device_status(stream), "status")
    got = as_bits(recv).reshape(n, n, count)
    host_in = np.stack([synth.host_buffer(dist, seed, x, count) for x in range(n)])
    return got, host_in


def run_rs_modes(n, count, dtype, seed, modes, dist=None):
    """Fill the inputs once, run the reduce-scatter in each execution mode
    (fresh, poisoned receive buffers each time) and return {mode: (N, count)
    host array} in the oracle's conventions."""
    dist = dist or DIST[dtype]
    dev = torch.device("cuda:0")
    send = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
    fill_ranks(send, dist, seed)
    recv = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
    stream = torch.cuda.current_stream()
    outs = {}
    for mode in modes:
        log(f"[gpu] reduce-scatter n={n} count={count} dtype={dtype} seed={seed:#x} mode={mode} (full output)")
        recv.view(torch.uint8).fill_(0x7F)
        pat.check(pat.pat_set_exec_mode(mode))
        pat.check(pat.pat_reducescatter(list(send), list(recv), count, dtype, pat.PAT_SUM, n, stream), "rs")
        pat.check(pat.pat_check_device_status(stream), "status")
        outs[mode] = as_bits(recv)
    del send, recv
    return outs


def compare_rs_full(outs, n, count, dtype, dist, seed, max_elems=1 << 25):
    """Every output element of every destination chunk against the threaded
    C++ oracle, which regenerates the inputs from the seed and streams over
    blocks of destination chunks: int32 bit-exact against the wrapped plain
    sum; float32 / bf16 bit-exact against the PAT association and within
    1e-5 / 1e-2 * sum|v| of the fp64 plain sum."""
    block = max(1, max_elems // max(count, 1))
    tol = 1e-5 if dtype == "float32" else 1e-2
    width = {"int32": np.uint32, "float32": np.uint32, "bfloat16": np.uint16}[dtype]
    for r0 in range(0, n, block):
        r1 = min(n, r0 + block)
        exp = native.reducescatter(dtype, n, count, dist=dist, seed=seed, r0=r0, r1=r1)
        for mode, got in outs.items():
            g = got[r0:r1]
            mism = int(np.count_nonzero(g.view(width) != exp["pat"].view(width)))
            assert mism == 0, f"{mode}: {mism} elements of chunks {r0}..{r1 - 1} differ from the PAT-order oracle"
            if dtype == "int32":
                wrapped = (exp["sum"].astype(np.int64) & 0xFFFFFFFF).astype(np.uint32).view(np.int32)
                assert (g == wrapped).all(), mode
                continue
            val = g.astype(np.float64) if dtype == "float32" else D.bf16_bits_to_f32(g).astype(np.float64)
            bad = int(np.count_nonzero(np.abs(val - exp["sum"]) > tol * exp["abs"]))
            assert bad == 0, f"{mode}: {bad} elements of chunks {r0}..{r1 - 1} outside {tol} of the fp64 sum"
    log(f"[gpu]   every element of {n} x {count} matches the oracle ({', '.join(outs)})")


# ---------------------------------------------------------------------------
# The generator itself: device fill == host twin
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dist", ["int32_pm2p20", "f32_pm1", "f32_normal", "bf16_normal"])
def test_device_fill_matches_host_twin(dist):
    log(f"[gpu] synth fill {dist}")
    dt = {"int32_pm2p20": torch.int32, "f32_pm1": torch.float32, "f32_normal": torch.float32,
          "bf16_normal": torch.bfloat16}[dist]
    buf = torch.empty(100003, dtype=dt, device="cuda:0")
    synth.fill(buf, dist, 0x1234, 7)
    want = synth.host_buffer(dist, 0x1234, 7, 100003)
    got = as_bits(buf)
    np.testing.assert_array_equal(got.view(want.dtype), want)


# ---------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
def test_workload1_rs_int32_n6(mode):
    n, count, seed = 6, 1024, 0x5041541
    got = run_rs(n, count, "int32", seed, mode=mode)
    check_rs(got, host_rs_inputs(n, count, "int32_pm2p20", seed), "int32", 0)


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
def test_workload2_ag_bf16_n24(mode):
    n, count, seed = 24, 32768, 0x5041542
    st, info = pat.pat_plan_info(pat.PAT_ALLGATHER, n, count, "bfloat16")
    assert info["slot_dims"] <= 5 and info["steps"] == 5  # ceil(log2 24)
    got, host_in = run_ag(n, count, "bfloat16", seed, mode=mode)
    np.testing.assert_array_equal(got, D.allgather(host_in))


def test_workload3_rs_f32_n64_every_element():
    """Workload 3 at its full size (N = 64, 1 MiB output chunks): every output
    element of every destination, in all four execution modes."""
    n, count, seed = 64, 262144, 0x5041543
    outs = run_rs_modes(n, count, "float32", seed, ["stream", "graph", "persistent", "dataflow"])
    compare_rs_full(outs, n, count, "float32", "f32_normal", seed)


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
def test_workload4_small_chunks_n1000(mode):
    """The small-size regime (N = 1000, 64 fp32 per chunk) as the benchmark
    runs it (AUTO fusion: 10 steps in 3 launches in stream and graph modes):
    the all-gather's whole output against the definition, and every one of the
    reduce-scatter's 1000 x 64 outputs bit-exact against the PAT order and
    within 1e-5 of the fp64 sum."""
    n, count, seed = 1000, 64, 0x5041544
    assert pat.pat_get_top_fusion() == pat.PAT_FUSION_AUTO
    st, info = pat.pat_plan_info(pat.PAT_ALLGATHER, n, count, "float32")
    assert info["steps"] == 10 and info["launches_per_op"] == 3
    got, host_in = run_ag(n, count, "float32", seed, mode=mode, dist="f32_pm1")
    assert (got == host_in[None, :, :]).all()
    outs = run_rs_modes(n, count, "float32", seed + 100, [mode], dist="f32_pm1")
    compare_rs_full(outs, n, count, "float32", "f32_pm1", seed + 100)


def test_workload5_rs_bf16_n128_every_element():
    """Workload 5 at its full size (N = 128, bf16 inputs, 4 MiB output chunks,
    64 GiB of send buffers): every one of the 128 x 2,097,152 outputs, in
    stream, graph and dataflow modes, bit-exact against the PAT order and
    within 1e-2 of the fp64 sum."""
    n, count, seed = 128, 2 * MIB, 0x5041545
    outs = run_rs_modes(n, count, "bfloat16", seed, ["stream", "graph", "dataflow"])
    pat.check(pat.pat_finalize())
    torch.cuda.empty_cache()
    compare_rs_full(outs, n, count, "bfloat16", "bf16_normal", seed)


@pytest.mark.parametrize("mode", ["stream", "graph"])
def test_workload7_ag_f32_n128_every_element(mode):
    """The bandwidth-regime all-gather at its benchmarked size (N = 128, 1 MiB
    chunks, 16 GiB of receive buffers): every element of every receive buffer
    against the definition, the concatenation of the host twin of the inputs
    (compared on the device, one receive buffer at a time)."""
    n, count, seed = 128, 262144, 0x5041547
    log(f"[gpu] all-gather n={n} count={count} float32 seed={seed:#x} mode={mode} (every element)")
    dev = torch.device("cuda:0")
    send = torch.empty((n, count), dtype=torch.float32, device=dev)
    fill_ranks(send, "f32_normal", seed)
    recv = torch.empty((n, n * count), dtype=torch.float32, device=dev)
    recv.view(torch.uint8).fill_(0xA5)
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    pat.check(pat.pat_allgather(list(send), list(recv), count, "float32", n, stream), "ag")
    pat.check(pat.pat_check_device_status(stream), "status")
    host_in = np.stack([synth.host_buffer("f32_normal", seed, x, count) for x in range(n)])
    want = torch.from_numpy(host_in.view(np.int32).reshape(-1)).to(dev)
    got = recv.view(torch.int32)
    bad = [r for r in range(n) if not torch.equal(got[r], want)]
    assert not bad, f"receive buffers {bad[:8]} differ from the concatenation"
    del send, recv, want, got
    pat.check(pat.pat_finalize())
    torch.cuda.empty_cache()


def test_maximum_rank_count():
    """N = 65536, the largest rank count the library accepts, with one-element
    chunks (16 GiB of rank buffers per collective, 128 KiB of slots per rank,
    16 steps).  The oracle's executors are quadratic in N, so outputs are
    sampled: the all-gather at 200 000 (receiver, chunk) pairs against the
    definition; the reduce-scatter at 48 destination ranks, int32 against the
    wrapped plain sum and float32 bit-exact against the closed form of the
    reversed trees (pinned to the oracle on small N) and within 1e-5 of the
    plain sum."""
    n, seed = 65536, 0x6A55
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode("stream"))
    stream = torch.cuda.current_stream()
    rng = np.random.default_rng(11)

    log(f"[gpu] all-gather n={n} count=1 int32 seed={seed:#x} (maximum rank count)")
    send = torch.empty((n, 1), dtype=torch.int32, device=dev)
    fill_ranks(send, "int32_pm2p20", seed)
    recv = torch.empty((n, n), dtype=torch.int32, device=dev)
    recv.view(torch.uint8).fill_(0xA5)
    pat.check(pat.pat_allgather(list(send), list(recv), 1, "int32", n, stream), "ag")
    pat.check(pat.pat_check_device_status(stream), "status")
    xs = np.unique(np.concatenate([[0, 1, n - 1], rng.integers(0, n, 2000)]))
    want = {int(x): synth.host_values("int32_pm2p20", seed, int(x), np.zeros(1, dtype=np.uint64))[0] for x in xs}
    xx = rng.choice(xs, 200000)
    rr = rng.integers(0, n, 200000)
    got = recv.view(-1)[torch.as_tensor(rr * n + xx, device=dev)].cpu().numpy()
    np.testing.assert_array_equal(got, np.array([want[int(x)] for x in xx], dtype=np.int32))
    del send, recv
    pat.check(pat.pat_finalize())
    torch.cuda.empty_cache()

    R = np.unique(np.concatenate([[0, 1, n - 1], rng.integers(0, n, 45)]))
    q = np.arange(n)
    for dtype, dist in (("int32", "int32_pm2p20"), ("float32", "f32_normal")):
        log(f"[gpu] reduce-scatter n={n} count=1 {dtype} seed={seed:#x} (maximum rank count)")
        send = torch.empty((n, n), dtype=TORCH[dtype], device=dev)
        fill_ranks(send, dist, seed)
        out = torch.empty((n, 1), dtype=TORCH[dtype], device=dev)
        pat.check(pat.pat_reducescatter(list(send), list(out), 1, dtype, pat.PAT_SUM, n, stream), "rs")
        pat.check(pat.pat_check_device_status(stream), "status")
        got = as_bits(out[torch.as_tensor(R, device=dev), 0])
        # vals[x, k]: rank x's contribution to destination R[k]
        vals = np.stack([synth.host_values(dist, seed, x, R.astype(np.uint64)) for x in range(n)])
        if dtype == "int32":
            want = (vals.astype(np.int64).sum(axis=0) & 0xFFFFFFFF).astype(np.uint32).view(np.int32)
            np.testing.assert_array_equal(got, want)
        else:
            # tree position q of destination R is rank R + q
            v = vals[(R[None, :] + q[:, None]) % n, np.arange(len(R))[None, :]]
            want = opat.reversed_tree_sum(v, n, lambda a, b: (a + b).astype(np.float32))
            np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))
            exact = vals.astype(np.float64).sum(axis=0)
            scale = np.abs(vals.astype(np.float64)).sum(axis=0)
            assert (np.abs(got.astype(np.float64) - exact) <= 1e-5 * scale).all()
        del send, out
        pat.check(pat.pat_finalize())
        torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Sweeps: rank counts, ragged sizes, budgets (aggregation levels, pieces), modes
# ---------------------------------------------------------------------------

SWEEP_N = [2, 3, 5, 7, 8, 13, 16, 33]


@pytest.mark.parametrize("mode", ["stream", "graph"])
@pytest.mark.parametrize("n", SWEEP_N)
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
@pytest.mark.parametrize("count", [1, 17, 1000, 4104])
def test_sweep_default_budget(n, dtype, count, mode):
    seed = 1000 * n + count
    got, host_in = run_ag(n, count, dtype, seed, mode=mode)
    np.testing.assert_array_equal(got, D.allgather(host_in))
    got = run_rs(n, count, dtype, seed + 1, mode=mode)
    check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
             oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))


@pytest.mark.parametrize("n", [5, 8, 13, 33])
@pytest.mark.parametrize("budget", [4096, 16384, 65536])
@pytest.mark.parametrize("mode", ["persistent", "graph", "stream", "dataflow"])
def test_sweep_budgets_and_modes(n, budget, mode):
    count = 4104  # float32: 16416-byte chunks, so 4096 B forces pieces and a ragged last piece
    pat.check(pat.pat_set_buffer_bytes(budget))
    try:
        for dtype in ("float32", "bfloat16"):
            seed = 7 * n + budget
            got, host_in = run_ag(n, count, dtype, seed, mode=mode)
            np.testing.assert_array_equal(got, D.allgather(host_in))
            got = run_rs(n, count, dtype, seed + 1, mode=mode)
            check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
                     oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))


@pytest.mark.parametrize("count", [1000, 1001, 1004])  # aligned; partial last vectors; bf16 RS 4-element vectors
@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
@pytest.mark.parametrize("n", [1, 6, 9])
def test_in_place(n, dtype, mode, count):
    """MPI-style in place (all-gather: send is chunk r of recv; reduce-scatter:
    recv is chunk r of send), where a reduce-scatter root's destination is its
    own input: with odd counts the rows are element-aligned and the relaxed
    kernels' partial last vectors store into the buffer they load from."""
    got, host_in = run_ag(n, count, dtype, 77 + n, inplace=True, mode=mode)
    np.testing.assert_array_equal(got, D.allgather(host_in))
    got = run_rs(n, count, dtype, 78 + n, inplace=True, mode=mode)
    check_rs(got, host_rs_inputs(n, count, DIST[dtype], 78 + n), dtype,
             oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))


def test_repeated_calls_reuse_plan_and_tables():
    """Same plan, different buffers on the second call (pointer tables re-uploaded)."""
    modes = ["persistent", "graph", "stream"]
    for rep in range(3):
        got, host_in = run_ag(12, 256, "float32", 500 + rep, mode=modes[rep])
        np.testing.assert_array_equal(got, D.allgather(host_in))
        got = run_rs(12, 256, "float32", 600 + rep, mode=modes[rep])
        check_rs(got, host_rs_inputs(12, 256, "f32_normal", 600 + rep), "float32",
                 oracle_t(pat.PAT_REDUCESCATTER, 12, 256, "float32"))


@pytest.mark.parametrize("mode", ["stream", "graph"])
@pytest.mark.parametrize("n", [6, 13, 33])
@pytest.mark.parametrize("budget", [4096, 65536])
def test_close_first_linear_order(n, budget, mode):
    count = 4104
    pat.check(pat.pat_set_buffer_bytes(budget))
    pat.check(pat.pat_set_linear_order("close"))
    try:
        for dtype in ("float32", "bfloat16", "int32"):
            seed = 31 * n + budget
            got, host_in = run_ag(n, count, dtype, seed, mode=mode)
            np.testing.assert_array_equal(got, D.allgather(host_in))
            got = run_rs(n, count, dtype, seed + 1, mode=mode)
            host = host_rs_inputs(n, count, DIST[dtype], seed + 1)
            if dtype == "int32":
                np.testing.assert_array_equal(got, D.reducescatter_sum(host, "int32"))
                continue
            t = oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype)
            pat_ref, _ = opat.reducescatter(host, t, dtype, "close")
            width = np.uint32 if dtype == "float32" else np.uint16
            assert (got.view(width) == pat_ref.view(width)).all()
    finally:
        pat.check(pat.pat_set_linear_order("far"))
        pat.check(pat.pat_set_buffer_bytes(0))


def test_persistent_barrier_timeout_is_reported_and_recovers():
    """Failure handling forced from the host: a 1 us limit on the persistent
    kernel's own bounded barrier wait.  Every workgroup still exits; the
    timeout is reported, and the next operation on the same plan is correct."""
    n, count, seed = 64, 262144, 0x77
    pat.check(pat.pat_set_barrier_timeout_us(1))
    try:
        dev = torch.device("cuda:0")
        send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        fill_ranks(send, "f32_normal", seed)
        recv = torch.empty((n, count), dtype=torch.float32, device=dev)
        pat.check(pat.pat_set_exec_mode("persistent"))
        stream = torch.cuda.current_stream()
        log("[gpu] persistent reduce-scatter with a 1 us barrier limit")
        pat.check(pat.pat_reducescatter(list(send), list(recv), count, "float32", pat.PAT_SUM, n, stream))
        assert pat.pat_check_device_status(stream) == pat.PAT_ERR_TIMEOUT
        assert pat.pat_check_device_status(stream) == pat.PAT_OK  # reported once, then cleared
        del send, recv
    finally:
        pat.check(pat.pat_set_barrier_timeout_us(0))
    sample = np.array([0, 5, 4096, count - 1])
    got = run_rs(n, count, "float32", seed, mode="persistent", sample=sample)
    check_rs(got, host_rs_inputs(n, count, "f32_normal", seed, sample), "float32",
             oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
@pytest.mark.parametrize("n,K", [(12, 2), (24, 5), (64, 3), (100, 6), (128, 7)])
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
def test_list_schedule_of_budget_aggregation(n, K, dtype, mode):
    """PAT_AGGREGATION_BUDGET with a budget of K chunks per step: the list
    schedule (fewer steps than the power-of-two one here) against the oracle,
    all-gather bit-exact, reduce-scatter bit-exact against the PAT order."""
    count, seed = 1000, 0x1157 + n * 7 + K
    pat.check(pat.pat_set_aggregation("budget"))
    try:
        for coll in ("ag", "rs"):
            slot = 4 if (coll == "rs" or dtype != "bfloat16") else 2
            pat.check(pat.pat_set_buffer_bytes(K * count * slot))
            code = pat.PAT_ALLGATHER if coll == "ag" else pat.PAT_REDUCESCATTER
            st, info = pat.pat_plan_info(code, n, count, dtype)
            assert info["list_schedule"] == 1, info
            if coll == "ag":
                got, host_in = run_ag(n, count, dtype, seed, mode=mode)
                np.testing.assert_array_equal(got, D.allgather(host_in))
            else:
                got = run_rs(n, count, dtype, seed, mode=mode)
                check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed), dtype, 0)
    finally:
        pat.check(pat.pat_set_aggregation("pow2"))
        pat.check(pat.pat_set_buffer_bytes(0))


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
@pytest.mark.parametrize("n,count,budget", [(5, 1000, 1024), (13, 4100, 4096), (33, 1001, 512)])
def test_pipelined_pieces(n, count, budget, dtype, mode, monkeypatch):
    """PAT_PIECE_PIPELINE=1: chunks larger than the budget in pieces of half
    the budget, alternating between the two halves of every slot, two pieces
    in flight (their steps one apart, in one launch) -- against the oracle,
    ragged last pieces included."""
    pat.check(pat.pat_finalize())
    monkeypatch.setenv("PAT_PIECE_PIPELINE", "1")
    pat.check(pat.pat_set_buffer_bytes(budget))
    seed = 0x9196 + n + count
    try:
        for coll in ("ag", "rs"):
            code = pat.PAT_ALLGATHER if coll == "ag" else pat.PAT_REDUCESCATTER
            st, info = pat.pat_plan_info(code, n, count, dtype)
            assert info["pieces"] >= 3
            if coll == "ag":
                got, host_in = run_ag(n, count, dtype, seed, mode=mode)
                np.testing.assert_array_equal(got, D.allgather(host_in))
            else:
                got = run_rs(n, count, dtype, seed, mode=mode)
                check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed), dtype, 0)
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))
        monkeypatch.delenv("PAT_PIECE_PIPELINE")
        pat.check(pat.pat_finalize())


def test_workload5_pipelined_pieces_every_element(monkeypatch):
    """Workload 5 with a 4 MiB budget (half of one float32 chunk): pieces of
    2 MiB alternating between the two slot halves, two in flight; every
    output element against the oracle, stream mode."""
    n, count, seed = 128, 2 * MIB, 0x5041545
    pat.check(pat.pat_finalize())
    monkeypatch.setenv("PAT_PIECE_PIPELINE", "1")
    pat.check(pat.pat_set_buffer_bytes(4 * MIB))
    try:
        st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, n, count, "bfloat16")
        assert info["pieces"] == 4 and info["launches_per_op"] == 2 * 127 + 1
        outs = run_rs_modes(n, count, "bfloat16", seed, ["stream"])
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))
        monkeypatch.delenv("PAT_PIECE_PIPELINE")
        pat.check(pat.pat_finalize())
        torch.cuda.empty_cache()
    compare_rs_full(outs, n, count, "bfloat16", "bf16_normal", seed)


def test_dataflow_wait_timeout_is_reported_and_recovers():
    """Failure handling forced from the host: a 1 us limit on the dataflow
    kernel's bounded waits for the buffers of earlier steps (1 MiB chunks:
    no step completes that fast).  Every workgroup still exits; the timeout
    is reported once, and the next operation on the same plan is correct."""
    n, count, seed = 64, 262144, 0x78
    pat.check(pat.pat_set_barrier_timeout_us(1))
    try:
        dev = torch.device("cuda:0")
        send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        fill_ranks(send, "f32_normal", seed)
        recv = torch.empty((n, count), dtype=torch.float32, device=dev)
        pat.check(pat.pat_set_exec_mode("dataflow"))
        stream = torch.cuda.current_stream()
        log("[gpu] dataflow reduce-scatter with a 1 us wait limit")
        pat.check(pat.pat_reducescatter(list(send), list(recv), count, "float32", pat.PAT_SUM, n, stream))
        assert pat.pat_check_device_status(stream) == pat.PAT_ERR_TIMEOUT
        assert pat.pat_check_device_status(stream) == pat.PAT_OK
        del send, recv
    finally:
        pat.check(pat.pat_set_barrier_timeout_us(0))
    outs = run_rs_modes(n, count, "float32", seed, ["dataflow"])
    compare_rs_full(outs, n, count, "float32", "f32_normal", seed)


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
def test_back_to_back_calls_with_new_buffers_no_host_sync(mode):
    """Three operations on one plan, each with its own buffers, queued without
    any host synchronisation: the pointer tables are re-staged each call while
    the previous call may still be running."""
    n, count = 11, 2048
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    sends, recvs = [], []
    for rep in range(3):
        send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        fill_ranks(send, "f32_normal", 900 + rep)
        recv = torch.empty((n, count), dtype=torch.float32, device=dev)
        sends.append(send)
        recvs.append(recv)
    log(f"[gpu] three queued reduce-scatters, mode={mode}")
    for rep in range(3):
        pat.check(pat.pat_reducescatter(list(sends[rep]), list(recvs[rep]), count, "float32", pat.PAT_SUM, n,
                                        stream))
    pat.check(pat.pat_check_device_status(stream))
    for rep in range(3):
        check_rs(as_bits(recvs[rep]), host_rs_inputs(n, count, "f32_normal", 900 + rep), "float32",
                 oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))


def test_plan_cache_is_bounded_and_evicts_safely():
    """With a 1-byte cap every new plan releases the previous one, after its
    last operation; results stay exact, and an evicted shape is rebuilt."""
    os.environ["PAT_PLAN_CACHE_BYTES"] = "1"
    try:
        pat.check(pat.pat_finalize())
        for i, count in enumerate([4096, 8192, 16384, 4096]):
            got = run_rs(16, count, "float32", 1234 + i)
            st, plans, nbytes = pat.pat_cache_stats()
            assert st == pat.PAT_OK and plans == 1 and nbytes > 0
            check_rs(got, host_rs_inputs(16, count, "f32_normal", 1234 + i), "float32",
                     oracle_t(pat.PAT_REDUCESCATTER, 16, count, "float32"))
    finally:
        os.environ.pop("PAT_PLAN_CACHE_BYTES", None)
        pat.check(pat.pat_finalize())


# ---------------------------------------------------------------------------
# Fused steps: one workgroup per (tree, tile) runs the top t steps (at full
# aggregation, every step)
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("mode", ["stream", "graph"])
@pytest.mark.parametrize("fusion", ["on", "off"])
@pytest.mark.parametrize("n", [4, 6, 13, 33, 100])
@pytest.mark.parametrize("count", [17, 1000, 20004])
def test_top_fusion_on_and_off(n, count, fusion, mode):
    # 20004 float32 elements: three tiles of the fused kernel, the last one ragged
    pat.check(pat.pat_set_top_fusion(fusion))
    try:
        for dtype in ("int32", "float32", "bfloat16"):
            if count == 20004 and n == 100 and dtype != "float32":
                continue  # keep the case small; the float32 run covers the shape
            seed = 31 * n + count + (fusion == "on")
            got, host_in = run_ag(n, count, dtype, seed, mode=mode)
            np.testing.assert_array_equal(got, D.allgather(host_in))
            got = run_rs(n, count, dtype, seed + 1, mode=mode)
            check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
                     oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))


@pytest.mark.parametrize("n,count,dtype", [(1000, 64, "float32"), (24, 32768, "bfloat16"), (64, 65536, "float32"),
                                           (37, 1001, "bfloat16")])
def test_top_fusion_is_bit_identical_to_step_kernels(n, count, dtype):
    """Same edges, same order of additions per element: fused and per-step
    execution give the same bits, for both collectives."""
    seed = 0x70F + n
    outs = {}
    for fusion in ("on", "off", "auto"):
        pat.check(pat.pat_set_top_fusion(fusion))
        try:
            ag, _ = run_ag(n, count, dtype, seed, mode="stream")
            rs = run_rs(n, count, dtype, seed + 1, mode="stream")
        finally:
            pat.check(pat.pat_set_top_fusion("auto"))
        outs[fusion] = (ag, rs)
    for fusion in ("on", "auto"):
        np.testing.assert_array_equal(outs[fusion][0], outs["off"][0])
        np.testing.assert_array_equal(outs[fusion][1], outs["off"][1])
    # and all of them against the oracle
    host_in = np.stack([synth.host_buffer(DIST[dtype], seed, x, count) for x in range(n)])
    np.testing.assert_array_equal(outs["off"][0], D.allgather(host_in))
    compare_rs_full({"off": outs["off"][1]}, n, count, dtype, DIST[dtype], seed + 1)


@pytest.mark.parametrize("n,count,dtype", [(1000, 64, "float32"), (24, 32768, "bfloat16"), (6, 1024, "int32"),
                                           (37, 1001, "bfloat16"), (129, 300, "float32")])
def test_tree_edge_cache_is_bit_identical(n, count, dtype, monkeypatch):
    """The fused launch's LDS edge cache (on by default; PAT_TREE_EDGE_CACHE=0
    turns it off) changes where lanes find their edges, not what they move:
    the same bits with and without it, for both collectives, and the
    oracle's."""
    seed = 0xEC0 + n
    outs = {}
    for flag in ("0", "1"):
        monkeypatch.setenv("PAT_TREE_EDGE_CACHE", flag)
        ag, host_in = run_ag(n, count, dtype, seed, mode="stream")
        rs = run_rs(n, count, dtype, seed + 1, mode="stream")
        outs[flag] = (ag, rs)
    np.testing.assert_array_equal(outs["1"][0], outs["0"][0])
    np.testing.assert_array_equal(outs["1"][1], outs["0"][1])
    np.testing.assert_array_equal(outs["1"][0], D.allgather(host_in))
    compare_rs_full({"cache": outs["1"][1]}, n, count, dtype, DIST[dtype], seed + 1)


def _max_chunks(n, t):
    return max(len(P) for _, P in opat.schedule(n, t))


def _span_cases():
    """(count, n, span) with a distinct aggregation level for the span: N = 3
    reaches full aggregation on the budget of span 4, so it has no span-4
    case; N = 1000 keeps to the smaller counts."""
    return [(count, n, span) for count in (5, 300, 4100) for n in (3, 5, 8, 9, 24, 31, 65, 129, 1000)
            for span in (2, 4) if (n, span) != (3, 4) and not (n == 1000 and count == 4100)]


@pytest.mark.parametrize("count,n,span", _span_cases())
def test_whole_schedule_fused_up_to_span_4(n, count, span):
    """With sub-trees of span 2 (full aggregation) or 4 every step joins the
    fused launch, the linear part included: one launch per operation, the
    oracle's results, and the same bits as one kernel per step."""
    L = opat.ceil_log2(n)
    t = L - (1 if span == 2 else 2)
    assert t >= 0
    seed = 0xF0 + 7 * n + count + span
    ran = 0
    try:
        for dtype in ("int32", "float32", "bfloat16"):
            if n == 1000 and dtype != "float32":
                continue  # keep the case small; the float32 run covers the shape
            for coll in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER):
                slot = 4 if (coll == pat.PAT_REDUCESCATTER or dtype != "bfloat16") else 2
                pat.check(pat.pat_set_buffer_bytes(_max_chunks(n, t) * count * slot))
                st, info = pat.pat_plan_info(coll, n, count, dtype)
                assert st == pat.PAT_OK
                if info["t"] != t or info["steps"] < 2:
                    continue  # truncation let this budget reach the next level
                outs = {}
                for fusion in ("on", "off"):
                    pat.check(pat.pat_set_top_fusion(fusion))
                    _, info = pat.pat_plan_info(coll, n, count, dtype)
                    assert info["fused_steps"] == (info["steps"] if fusion == "on" else 0)
                    mode = "graph" if n == 24 else "stream"
                    if coll == pat.PAT_ALLGATHER:
                        outs[fusion] = run_ag(n, count, dtype, seed, mode=mode)
                    else:
                        outs[fusion] = run_rs(n, count, dtype, seed + 1, mode=mode)
                pat.check(pat.pat_set_top_fusion("auto"))
                if coll == pat.PAT_ALLGATHER:
                    got, host_in = outs["on"]
                    np.testing.assert_array_equal(got, D.allgather(host_in))
                    np.testing.assert_array_equal(got, outs["off"][0])
                else:
                    check_rs(outs["on"], host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
                             oracle_t(coll, n, count, dtype))
                    np.testing.assert_array_equal(outs["on"], outs["off"])
                ran += 1
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))
        pat.check(pat.pat_set_buffer_bytes(0))
    assert ran > 0


def test_workload3_and_2_with_fusion_forced_on():
    pat.check(pat.pat_set_top_fusion("on"))
    try:
        n, count, seed = 64, 262144, 0x5041543
        rng = np.random.default_rng(3)
        sample = np.unique(np.concatenate([[0, 1, 8191, 8192, count - 1], rng.integers(0, count, 600)]))
        got = run_rs(n, count, "float32", seed, sample=sample, mode="stream")
        check_rs(got, host_rs_inputs(n, count, "f32_normal", seed, sample), "float32",
                 oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))
        got, host_in = run_ag(24, 32768, "bfloat16", 0x5041542, mode="graph")
        np.testing.assert_array_equal(got, D.allgather(host_in))
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))


def test_graph_mode_follows_fusion_changes_on_one_plan():
    """Graph mode keeps a captured graph per fused range: switching the fusion
    setting between calls on the same plan replays the matching graph, and
    every replay gives the same bits."""
    n, count, seed = 1000, 64, 0x6A11
    outs = []
    try:
        for fusion in ("on", "auto", "off", "on", "auto"):
            pat.check(pat.pat_set_top_fusion(fusion))
            outs.append(run_rs(n, count, "float32", seed, mode="graph", dist="f32_pm1"))
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])
    compare_rs_full({"graph": outs[0]}, n, count, "float32", "f32_pm1", seed)


@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
def test_tensor_wrappers(dtype):
    """pat.allgather / pat.reducescatter on 2-D tensors (one row per rank) and
    on lists of rows give the oracle's results."""
    n, count, seed = 9, 1000, 0x7E5
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode("stream"))
    send = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
    fill_ranks(send, DIST[dtype], seed)
    recv = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
    pat.allgather(send, recv)
    host_in = np.stack([synth.host_buffer(DIST[dtype], seed, x, count) for x in range(n)])
    np.testing.assert_array_equal(as_bits(recv).reshape(n, n, count), D.allgather(host_in))
    rs_in = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
    fill_ranks(rs_in, DIST[dtype], seed + 1)
    out = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
    pat.reducescatter(list(rs_in), list(out))
    check_rs(as_bits(out), host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
             oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))


def test_tensor_wrappers_default_to_the_current_stream():
    """Inside ``torch.cuda.stream(side)`` the wrappers run on `side` (torch's
    current stream), after the side-stream work that produced their inputs,
    and before the side-stream work that reads their outputs."""
    n, count, seed = 7, 200003, 0x51DE
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode("stream"))
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=dev)  # default priority
    with torch.cuda.stream(side):
        send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        fill_ranks(send, "f32_normal", seed)  # queued on the side stream
        out = torch.empty((n, count), dtype=torch.float32, device=dev)
        pat.reducescatter(send, out)
        snap = out.clone()  # side-stream reader of the result
        ag_in = torch.empty((n, count), dtype=torch.float32, device=dev)
        fill_ranks(ag_in, "f32_normal", seed + 1)
        ag_out = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        pat.allgather(ag_in, ag_out)
        ag_snap = ag_out[:, -count:].clone()
    side.synchronize()
    log("[gpu] tensor wrappers on the current (side) stream")
    sample = np.array([0, 1, 4095, 4096, count - 1])
    host_in = host_rs_inputs(n, count, "f32_normal", seed, sample)
    check_rs(as_bits(snap)[:, sample], host_in, "float32", oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))
    want = np.stack([synth.host_buffer("f32_normal", seed + 1, x, count) for x in range(n)])
    np.testing.assert_array_equal(as_bits(ag_snap), np.broadcast_to(want[n - 1], (n, count)))


@pytest.mark.parametrize("n,count,dtype,coll", [(1000, 64, "float32", "rs"), (24, 32768, "bfloat16", "ag"),
                                                  (64, 4096, "float32", "rs"), (13, 1001, "bfloat16", "rs")])
def test_launch_trace_covers_every_launch(n, count, dtype, coll):
    """pat_trace_start / pat_trace_read: one event pair per kernel launch of
    the traced operations, in launch order, whose bytes add up to the plan's
    algorithmic bytes per operation; the traced results stay exact."""
    pat.check(pat.pat_set_exec_mode("stream"))
    code = pat.PAT_REDUCESCATTER if coll == "rs" else pat.PAT_ALLGATHER
    st, info = pat.pat_plan_info(code, n, count, dtype)
    launches = info["launches_per_op"]
    pat.check(pat.pat_trace_start(2 * launches + 1))
    seed = 0x7ACE + n
    if coll == "rs":
        got = run_rs(n, count, dtype, seed, mode="stream")
        got2 = run_rs(n, count, dtype, seed, mode="stream")
        check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed), dtype, oracle_t(code, n, count, dtype))
    else:
        got, host_in = run_ag(n, count, dtype, seed, mode="stream")
        got2, _ = run_ag(n, count, dtype, seed, mode="stream")
        np.testing.assert_array_equal(got, D.allgather(host_in))
    np.testing.assert_array_equal(got, got2)
    assert pat.pat_trace_read(1)[0] == pat.PAT_ERR_INVALID_ARGUMENT  # too small: stays armed
    st, rows = pat.pat_trace_read(2 * launches + 1)
    pat.check(st)
    assert len(rows) == 2 * launches
    for op in (rows[:launches], rows[launches:]):
        assert sum(r[1] for r in op) == pytest.approx(info["alg_bytes"], rel=1e-9)
        assert all(r[0] > 0 for r in op)
        assert [r[3] for r in op] == sorted(r[3] for r in op)  # launch order
        assert sum(r[2] for r in op) == (1 if info["fused_steps"] else 0)
    assert pat.pat_trace_read(4)[0] == pat.PAT_ERR_INVALID_ARGUMENT  # disarmed


@pytest.mark.parametrize("n,count,dtype,coll", [(1000, 64, "float32", "rs"), (1000, 64, "float32", "ag"),
                                                  (24, 32768, "bfloat16", "ag"), (6, 1024, "int32", "rs")])
def test_step_clock_of_fused_launches(n, count, dtype, coll, monkeypatch):
    """PAT_STEP_CLOCK=1: the fused kernel records, per workgroup, one stamp
    before its first step and one after each, never decreasing; the result
    stays exact; with the variable off nothing is recorded."""
    code = pat.PAT_REDUCESCATTER if coll == "rs" else pat.PAT_ALLGATHER
    st, info = pat.pat_plan_info(code, n, count, dtype)
    assert info["fused_steps"] >= 2
    pat.check(pat.pat_finalize())
    monkeypatch.setenv("PAT_STEP_CLOCK", "1")
    seed = 0xC10C + n
    try:
        if coll == "rs":
            got = run_rs(n, count, dtype, seed, mode="stream")
            check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed), dtype, oracle_t(code, n, count, dtype))
        else:
            got, host_in = run_ag(n, count, dtype, seed, mode="stream")
            np.testing.assert_array_equal(got, D.allgather(host_in))
        st, stamps, tpu = pat.pat_step_clock(code, n, count, dtype)
        pat.check(st, "pat_step_clock")
        assert stamps.shape[1] == info["fused_steps"] + 1 and stamps.shape[0] % n == 0
        assert (np.diff(stamps.astype(np.int64), axis=1) >= 0).all() and (stamps[:, 0] > 0).all()
        assert 1.0 <= tpu <= 10000.0
    finally:
        monkeypatch.delenv("PAT_STEP_CLOCK")
        pat.check(pat.pat_finalize())
    if coll == "rs":
        run_rs(n, count, dtype, seed, mode="stream")
    else:
        run_ag(n, count, dtype, seed, mode="stream")
    assert pat.pat_step_clock(code, n, count, dtype)[0] == pat.PAT_ERR_INVALID_ARGUMENT


def test_pointer_checks_follow_every_argument():
    """The per-pointer checks are skipped only for the exact pointer set a
    thread last validated with the same operation, rank count, count and
    dtype.  The same receive pointers with a doubled count overlap (rows are
    packed for the smaller count) and must be refused before any launch; the
    valid call still works before and after, and a one-entry change is
    checked again."""
    n, count, seed = 4, 64, 0x5EC
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode("stream"))
    stream = torch.cuda.current_stream()
    send = torch.empty((n, 2 * count), dtype=torch.float32, device=dev)
    fill_ranks(send, "f32_normal", seed)
    recv = torch.empty((n, n * count), dtype=torch.float32, device=dev)
    S, R = pat.pointer_array([send[x, :count] for x in range(n)]), pat.pointer_array(list(recv))
    want = np.stack([synth.host_buffer("f32_normal", seed, x, 2 * count)[:count] for x in range(n)])
    for attempt in range(2):
        for repeat in range(2):  # the second call takes the already-checked path
            recv.fill_(-1.0)
            pat.check(pat.pat_allgather(S, R, count, "float32", n, stream), "ag")
            got = as_bits(recv).reshape(n, n, count)
            for r in range(n):
                np.testing.assert_array_equal(got[r], want)
        # doubled count: receive rows of n * 2 * count elements overlap their neighbours
        assert pat.pat_allgather(S, R, 2 * count, "float32", n, stream) == pat.PAT_ERR_INVALID_ARGUMENT
        # a set that differs in one entry (rank 1's receive buffer inside rank 0's) is checked again
        bad = pat.pointer_array([recv[0].data_ptr()] + [recv[0].data_ptr() + 256] + [recv[r].data_ptr() for r in (2, 3)])
        assert pat.pat_allgather(S, bad, count, "float32", n, stream) == pat.PAT_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()


def _random_cases(k=100, seed=2026):
    """A fixed, seeded draw of configurations mixing every setting."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(k):
        n = int(rng.choice([2, 3, 5, 7, 12, 17, 31, 45, 64, 100, 129, 200]))
        dtype = str(rng.choice(["int32", "float32", "bfloat16"]))
        count = int(rng.choice([1, 3, 8, 33, 250, 1000, 2052]))
        budget = int(rng.choice([0, 64, 512, 4096, 65536]))  # 0: default; small budgets force pieces
        mode = str(rng.choice(["stream", "graph", "persistent", "dataflow"]))
        fusion = str(rng.choice(["auto", "on", "off"]))
        order = str(rng.choice(["far", "close"]))
        coll = str(rng.choice(["ag", "rs"]))
        cases.append((coll, n, count, dtype, budget, mode, fusion, order, int(rng.integers(1, 1 << 30))))
    return cases


@pytest.mark.parametrize("case", _random_cases(), ids=lambda c: "-".join(str(x) for x in c[:8]))
def test_random_configurations(case):
    """Seeded random mixes of rank count, size, dtype, buffer budget (pieces
    included), execution mode, fusion and linear order, against the oracle."""
    coll, n, count, dtype, budget, mode, fusion, order, seed = case
    pat.check(pat.pat_set_buffer_bytes(budget))
    pat.check(pat.pat_set_top_fusion(fusion))
    pat.check(pat.pat_set_linear_order(order))
    try:
        if coll == "ag":
            got, host_in = run_ag(n, count, dtype, seed, mode=mode)
            np.testing.assert_array_equal(got, D.allgather(host_in))
        else:
            got = run_rs(n, count, dtype, seed, mode=mode)
            check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed), dtype,
                     oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype), order)
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))
        pat.check(pat.pat_set_top_fusion("auto"))
        pat.check(pat.pat_set_linear_order("far"))


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
def test_caller_created_stream(mode):
    """The collectives run on the stream they are given, not only on the
    default one."""
    n, count, seed = 13, 3000, 0x57E
    dev = torch.device("cuda:0")
    send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
    fill_ranks(send, "f32_normal", seed)
    recv = torch.empty((n, count), dtype=torch.float32, device=dev)
    agin = torch.empty((n, count), dtype=torch.bfloat16, device=dev)
    fill_ranks(agin, "bf16_normal", seed + 1)
    agout = torch.empty((n, n * count), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    side = torch.cuda.Stream(device=dev)  # default priority
    pat.check(pat.pat_set_exec_mode(mode))
    log(f"[gpu] caller stream, mode={mode}")
    pat.check(pat.pat_reducescatter(list(send), list(recv), count, "float32", pat.PAT_SUM, n, side))
    pat.check(pat.pat_allgather(list(agin), list(agout), count, "bfloat16", n, side))
    pat.check(pat.pat_check_device_status(side))
    check_rs(as_bits(recv), host_rs_inputs(n, count, "f32_normal", seed), "float32",
             oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))
    host_in = np.stack([synth.host_buffer("bf16_normal", seed + 1, x, count) for x in range(n)])
    np.testing.assert_array_equal(as_bits(agout).reshape(n, n, count), D.allgather(host_in))


def test_two_host_threads_on_their_own_streams():
    """Two host threads issue collectives concurrently, each on its own stream
    and plan; the library serialises its host-side work and the device runs
    both streams at once."""
    import threading

    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode("stream"))
    jobs = [(9, 4000, 0x7A1), (17, 2500, 0x7A2)]
    bufs = []
    for n, count, seed in jobs:
        send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        fill_ranks(send, "f32_normal", seed)
        bufs.append((send, torch.empty((n, count), dtype=torch.float32, device=dev)))
    torch.cuda.synchronize()
    errors = []

    def worker(idx):
        try:
            n, count, _ = jobs[idx]
            send, recv = bufs[idx]
            s = torch.cuda.Stream(device=dev)
            S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))
            for _ in range(20):
                pat.check(pat.pat_reducescatter(S, R, count, "float32", pat.PAT_SUM, n, s))
            pat.check(pat.pat_check_device_status(s))
        except Exception as exc:  # reported by the main thread
            errors.append(exc)

    log("[gpu] two host threads")
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for (n, count, seed), (send, recv) in zip(jobs, bufs):
        check_rs(as_bits(recv), host_rs_inputs(n, count, "f32_normal", seed), "float32",
                 oracle_t(pat.PAT_REDUCESCATTER, n, count, "float32"))


def test_large_rank_count_n2049():
    """N = 2049 (L = 12, not a power of two), full aggregation, tiny chunks:
    int32 and float32 reduce-scatter and all-gather on the 128-bit path
    (4 elements) and the element path (3 elements), every output checked."""
    n = 2049
    got = run_rs(n, 4, "int32", 0x801, mode="stream")
    np.testing.assert_array_equal(got, D.reducescatter_sum(host_rs_inputs(n, 4, "int32_pm2p20", 0x801), "int32"))
    got = run_rs(n, 3, "float32", 0x802, mode="stream")
    host_in = host_rs_inputs(n, 3, "f32_normal", 0x802)
    exact = D.reducescatter_sum(host_in, "float32")
    scale = D.reducescatter_abs_sum(host_in, "float32")
    assert (np.abs(got.astype(np.float64) - exact) <= 1e-5 * scale).all()
    for count, dtype in ((3, "float32"), (8, "bfloat16")):
        got, host_in = run_ag(n, count, dtype, 0x803 + count, mode="stream")
        np.testing.assert_array_equal(got, D.allgather(host_in))
    torch.cuda.empty_cache()


@pytest.mark.parametrize("tile", ["7", "100"])
def test_top_fusion_with_odd_tiles(tile, monkeypatch):
    """The fused kernel with tiles that do not divide the chunk: many tiles
    per tree and a ragged last one, every dtype, both collectives."""
    monkeypatch.setenv("PAT_TREE_TILE", tile)
    pat.check(pat.pat_set_top_fusion("on"))
    try:
        for n, count in ((13, 1000), (33, 4104)):
            for dtype in ("int32", "float32", "bfloat16"):
                seed = 41 * n + count + int(tile)
                got, host_in = run_ag(n, count, dtype, seed, mode="stream")
                np.testing.assert_array_equal(got, D.allgather(host_in))
                got = run_rs(n, count, dtype, seed + 1, mode="stream")
                check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
                         oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))


@pytest.mark.parametrize("grain", ["1", "3", "7", "1000"])
def test_xcd_run_lengths(grain, monkeypatch):
    """The step kernels' XCD work order with run lengths that divide nothing:
    every work item is still done exactly once (the grid is padded to a
    multiple of 8 runs and the surplus workgroups have no item)."""
    monkeypatch.setenv("PAT_XCD_GRAIN", grain)
    pat.check(pat.pat_finalize())  # the run length is fixed when a plan is made
    try:
        for n, count in ((13, 1000), (7, 20004), (33, 17)):
            for dtype in ("int32", "float32", "bfloat16"):
                seed = 53 * n + count + int(grain)
                got, host_in = run_ag(n, count, dtype, seed, mode="stream")
                np.testing.assert_array_equal(got, D.allgather(host_in))
                got = run_rs(n, count, dtype, seed + 1, mode="stream")
                check_rs(got, host_rs_inputs(n, count, DIST[dtype], seed + 1), dtype,
                         oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))
    finally:
        monkeypatch.delenv("PAT_XCD_GRAIN")
        pat.check(pat.pat_finalize())


# ---------------------------------------------------------------------------
# Relaxed 128-bit kernels: element-aligned buffers, partial last vectors
# ---------------------------------------------------------------------------

def _rows(flat, n, length, skew):
    """n rows of `length` elements carved from one flat buffer, starting
    `skew` elements in: every row is element-aligned, most are not 16-byte
    aligned."""
    return [flat[skew + r * length: skew + (r + 1) * length] for r in range(n)]


@pytest.mark.parametrize("mode", ["stream", "graph", "persistent", "dataflow"])
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
def test_relaxed_vectors_at_element_offsets(dtype, mode):
    """Buffers one element past a 16-byte boundary, and counts just under,
    at and over one vector and one tile (a partial last vector that is the
    only vector, that closes a tile, that opens one), through the relaxed
    128-bit kernels, against the oracle; plan_info reports the path
    16-byte-aligned buffers take."""
    es = {"int32": 4, "float32": 4, "bfloat16": 2}[dtype]
    per = 16 // es  # elements per all-gather vector
    counts = [per - 1, per, per + 1, 2 * per + 3, 2047, 2049, 4100, 4096 * 2 // es - 1]
    dev = torch.device("cuda:0")
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    dist = DIST[dtype]
    for n in (5, 16):
        for count in counts:
            seed = 0xA11 + 31 * count + n
            log(f"[gpu] relaxed n={n} count={count} dtype={dtype} mode={mode}")
            # all-gather
            sflat = torch.empty(n * count + 1, dtype=TORCH[dtype], device=dev)
            rflat = torch.empty(n * n * count + 1, dtype=TORCH[dtype], device=dev)
            rflat.view(torch.uint8).fill_(0xA5)
            sends, recvs = _rows(sflat, n, count, 1), _rows(rflat, n, n * count, 1)
            for r in range(n):
                synth.fill(sends[r], dist, seed, r)
            pat.check(pat.pat_allgather(sends, recvs, count, dtype, n, stream), "ag")
            pat.check(pat.pat_check_device_status(stream), "status")
            got = as_bits(torch.stack(recvs)).reshape(n, n, count)
            host_in = np.stack([synth.host_buffer(dist, seed, x, count) for x in range(n)])
            np.testing.assert_array_equal(got, D.allgather(host_in))
            # the element before the skewed rows is untouched
            assert as_bits(rflat[:1]).view(np.uint8).tolist() == [0xA5] * es
            st, info = pat.pat_plan_info(pat.PAT_ALLGATHER, n, count, dtype)
            pat.check(st)
            assert info["vector_path"] == (0 if count < per else 1 if count % per == 0 else 2)
            # reduce-scatter
            sflat = torch.empty(n * n * count + 1, dtype=TORCH[dtype], device=dev)
            rflat = torch.empty(n * count + 1, dtype=TORCH[dtype], device=dev)
            rflat.view(torch.uint8).fill_(0x7F)
            sends, recvs = _rows(sflat, n, n * count, 1), _rows(rflat, n, count, 1)
            for r in range(n):
                synth.fill(sends[r], dist, seed + 1, r)
            pat.check(pat.pat_reducescatter(sends, recvs, count, dtype, pat.PAT_SUM, n, stream), "rs")
            pat.check(pat.pat_check_device_status(stream), "status")
            got = as_bits(torch.stack(recvs))
            check_rs(got, host_rs_inputs(n, count, dist, seed + 1), dtype,
                     oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype))
            assert as_bits(rflat[:1]).view(np.uint8).tolist() == [0x7F] * es
            st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, n, count, dtype)
            pat.check(st)
            # reduce-scatter vectors hold 4 elements (bf16: 8-byte inputs)
            want = 1 if count % 4 == 0 else 2 if count >= 4 else 0
            assert info["vector_path"] == want
            del sflat, rflat, sends, recvs


def _skewed_cases(k=60, seed=2027):
    """A fixed, seeded draw of skewed-buffer configurations."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(k):
        n = int(rng.choice([2, 3, 6, 9, 24, 64, 130]))
        dtype = str(rng.choice(["int32", "float32", "bfloat16"]))
        count = int(rng.choice([4, 7, 12, 64, 333, 1024, 2051, 4099]))
        budget = int(rng.choice([0, 100, 1000, 4096]))  # small budgets: pieces, each with its partial vector
        mode = str(rng.choice(["stream", "graph", "persistent", "dataflow"]))
        fusion = str(rng.choice(["auto", "on", "off"]))
        order = str(rng.choice(["far", "close"]))
        coll = str(rng.choice(["ag", "rs"]))
        skew = int(rng.integers(1, 8))
        cases.append((coll, n, count, dtype, budget, mode, fusion, order, skew, int(rng.integers(1, 1 << 30))))
    return cases


@pytest.mark.parametrize("case", _skewed_cases(), ids=lambda c: "-".join(str(x) for x in c[:9]))
def test_random_skewed_buffers(case):
    """Seeded random mixes with every buffer 1 to 7 elements past a 16-byte
    boundary (relaxed or element-wide kernels, pieces with partial last
    vectors), against the oracle."""
    coll, n, count, dtype, budget, mode, fusion, order, skew, seed = case
    dev = torch.device("cuda:0")
    dist = DIST[dtype]
    pat.check(pat.pat_set_buffer_bytes(budget))
    pat.check(pat.pat_set_top_fusion(fusion))
    pat.check(pat.pat_set_linear_order(order))
    pat.check(pat.pat_set_exec_mode(mode))
    stream = torch.cuda.current_stream()
    log(f"[gpu] skewed {case}")
    try:
        slen, rlen = (count, n * count) if coll == "ag" else (n * count, count)
        sflat = torch.empty(n * slen + skew, dtype=TORCH[dtype], device=dev)
        rflat = torch.empty(n * rlen + skew, dtype=TORCH[dtype], device=dev)
        rflat.view(torch.uint8).fill_(0x5A)
        sends, recvs = _rows(sflat, n, slen, skew), _rows(rflat, n, rlen, skew)
        for r in range(n):
            synth.fill(sends[r], dist, seed, r)
        if coll == "ag":
            pat.check(pat.pat_allgather(sends, recvs, count, dtype, n, stream), "ag")
            pat.check(pat.pat_check_device_status(stream), "status")
            got = as_bits(torch.stack(recvs)).reshape(n, n, count)
            host_in = np.stack([synth.host_buffer(dist, seed, x, count) for x in range(n)])
            np.testing.assert_array_equal(got, D.allgather(host_in))
        else:
            pat.check(pat.pat_reducescatter(sends, recvs, count, dtype, pat.PAT_SUM, n, stream), "rs")
            pat.check(pat.pat_check_device_status(stream), "status")
            check_rs(as_bits(torch.stack(recvs)), host_rs_inputs(n, count, dist, seed), dtype,
                     oracle_t(pat.PAT_REDUCESCATTER, n, count, dtype), order)
        assert (as_bits(rflat[:skew]).view(np.uint8) == 0x5A).all()
        del sflat, rflat, sends, recvs
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))
        pat.check(pat.pat_set_top_fusion("auto"))
        pat.check(pat.pat_set_linear_order("far"))


@pytest.mark.parametrize("case", [
    ("rs", 128, 2 * MIB - 1, "bfloat16", "stream"),
    ("rs", 128, 2 * MIB - 3, "bfloat16", "persistent"),
    ("rs", 64, 262144 - 1, "float32", "stream"),
    ("rs", 64, 262144 - 3, "int32", "stream"),
    ("ag", 128, 262144 - 1, "float32", "stream"),
    ("ag", 128, 524288 - 3, "bfloat16", "stream"),
], ids=lambda c: "-".join(str(x) for x in c))
def test_streaming_relaxed_kernels_full_size(case):
    """Odd counts at the benchmarked sizes: the relaxed kernels in their
    streaming (nontemporal) form, which only operations of 1e9 or more
    algorithmic bytes use, against the oracle at every output element (every
    chunk's partial last vector and the elements it overlaps included)."""
    coll, n, count, dtype, mode = case
    seed = 0x0DD0 + count
    dist = DIST[dtype]
    if coll == "rs":
        outs = run_rs_modes(n, count, dtype, seed, [mode])
        pat.check(pat.pat_finalize())
        torch.cuda.empty_cache()
        compare_rs_full(outs, n, count, dtype, dist, seed)
    else:
        dev = torch.device("cuda:0")
        log(f"[gpu] all-gather n={n} count={count} {dtype} seed={seed:#x} (full size, odd, every element)")
        send = torch.empty((n, count), dtype=TORCH[dtype], device=dev)
        fill_ranks(send, dist, seed)
        recv = torch.empty((n, n * count), dtype=TORCH[dtype], device=dev)
        recv.view(torch.uint8).fill_(0xA5)
        pat.check(pat.pat_set_exec_mode(mode))
        stream = torch.cuda.current_stream()
        pat.check(pat.pat_allgather(list(send), list(recv), count, dtype, n, stream), "ag")
        pat.check(pat.pat_check_device_status(stream), "status")
        host_in = np.stack([synth.host_buffer(dist, seed, x, count) for x in range(n)])
        iview = torch.int16 if dtype == "bfloat16" else torch.int32
        want = torch.from_numpy(host_in.view(np.int16 if dtype == "bfloat16" else np.int32).reshape(-1)).to(dev)
        got = recv.view(iview)
        bad = [r for r in range(n) if not torch.equal(got[r], want)]
        assert not bad, f"receive buffers {bad[:8]} differ from the concatenation"
        del send, recv, want, got
    pat.check(pat.pat_finalize())
    torch.cuda.empty_cache()
