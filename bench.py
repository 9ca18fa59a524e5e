"""Benchmark: PAT reduce-scatter of 128 virtual ranks on one MI355X.

Workload (the bandwidth-roofline case): reduce-scatter (sum), N = 128
virtual ranks, bf16 inputs N(0,1) from seed 0x5041545, float32 partial sums,
a 4 MiB output chunk (2,097,152 bf16) per rank -- 64 GiB of rank send buffers
resident in HBM.  One "step" = one whole reduce-scatter over all 128 ranks.

Prints one JSON line:
* value      -- aggregate bus bandwidth, N * (N-1) * C / t  (nccl-tests busBW
                summed over the N virtual ranks; the per-rank figure is
                bus_gbps_per_rank); t = the mean of the timed operations, each
                bracketed by its own HIP events (the median is reported too)
* roofline   -- the dominant kernel's own rate: the algorithmic bytes of its
                launches / their durations, from a HIP event pair recorded on
                the kernels' stream around every launch of the first three
                timed operations; against the 8 TB/s HBM3E peak; traffic from
                the committed rocprofv3 counter summary when it matches the
                current kernel source
* cpu_baseline -- the CPU oracle timed in the same process: the threaded C++
                oracle over the whole operation on every host CPU, inputs
                regenerated from the seed (reduce-scatter: PAT association and
                fp64 plain sum; all-gather: concatenation, repeated for at least
                --cpu-seconds); in the same unit

python bench.py [--steps K] [--warmup W] [--mode persistent|graph|stream]
                [--workload 1..7] [--cpu-seconds S] [--no-cpu-baseline]
(workloads 6 and 7: the all-gather in the small-size and bandwidth regimes)
"""

import argparse
import hashlib
import math
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "bus GB/s and % of HBM peak for PAT AG/RS; small-size latency µs"

WORKLOADS = {
    # id: (collective, N, count, dtype, distribution, seed, description)
    1: ("rs", 6, 1024, "int32", "int32_pm2p20", 0x5041541,
        "PAT reduce-scatter (sum), N=6 virtual ranks, int32 U[-2^20,2^20], 1024-element output chunk"),
    2: ("ag", 24, 32768, "bfloat16", "bf16_normal", 0x5041542,
        "PAT all-gather, N=24 virtual ranks, bf16 N(0,1), 32768-element (64 KiB) chunk per rank"),
    3: ("rs", 64, 262144, "float32", "f32_normal", 0x5041543,
        "PAT reduce-scatter (sum), N=64 virtual ranks, fp32 N(0,1), 262144-element (1 MiB) output chunk"),
    4: ("rs", 1000, 64, "float32", "f32_pm1", 0x5041544,
        "PAT reduce-scatter (sum), N=1000 virtual ranks, fp32 U[-1,1), 64-element (256 B) output chunk"),
    5: ("rs", 128, 2097152, "bfloat16", "bf16_normal", 0x5041545,
        "PAT reduce-scatter (sum), N=128 virtual ranks, bf16 N(0,1) in / fp32 accumulation, "
        "2097152-element (4 MiB) output chunk per rank, 64 GiB of rank buffers in HBM"),
    # the all-gather of the small-size regime (workload 4's other collective)
    6: ("ag", 1000, 64, "float32", "f32_pm1", 0x5041544,
        "PAT all-gather, N=1000 virtual ranks, fp32 U[-1,1), 64-element (256 B) chunk per rank"),
    # the all-gather in the bandwidth regime (1 MiB chunks, 16 GiB of receive buffers)
    7: ("ag", 128, 262144, "float32", "f32_normal", 0x5041547,
        "PAT all-gather, N=128 virtual ranks, fp32 N(0,1), 262144-element (1 MiB) chunk per rank"),
}

KERNEL_SOURCES = ["paper_2506_20252_amd/csrc/kernels.hip", "paper_2506_20252_amd/csrc/kernels.hpp",
                  "paper_2506_20252_amd/csrc/device_types.hpp"]


def _code_only(text):
    """C/C++ source without comments and whitespace: what the compiler sees
    (string and character literals kept intact)."""
    out, i, n = [], 0, len(text)
    while i < n:
        ch = text[i]
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        elif ch in "\"'":
            j = i + 1
            while j < n and text[j] != ch:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            if not ch.isspace():
                out.append(ch)
            i += 1
    return "".join(out)


def kernel_source_hash():
    """Hash of the kernel sources' code (comments and whitespace ignored), so
    that counter summaries stay valid across comment edits only."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def committed_traffic(workload_id, mode, kernel):
    """HBM-side bytes per launch of `kernel` (step_kernel / tree_kernel) from
    the committed counter summary, if it was taken on the current kernel
    source; else None.  Stream and graph modes launch the same kernels; the
    persistent kernel has no summary."""
    if mode == "persistent":
        return None
    kind = "tree_kernel" if kernel.startswith("tree_kernel") else "step_kernel"
    path = os.path.join(ROOT, "profiles", f"traffic_{kind}_workload{workload_id}.txt")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_source_hash:\s*(\w+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_source_hash():
        return None
    return float(m_bytes.group(1))


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            return next((line.split(":", 1)[1].strip() for line in f if line.startswith("model name")), "")
    except OSError:
        return ""


def cpu_baseline_rs(wid):
    """The threaded C++ oracle over the whole reduce-scatter: every destination
    chunk and every element, the PAT association (float32, or int32) and the
    fp64 plain sum, inputs regenerated from the seed, on every CPU this process
    may use.  Streams over blocks of destination chunks, so that nothing the
    size of the send buffers sits in host memory."""
    import numpy as np  # noqa: F401

    from oracle import native

    coll, n, count, dtype, dist, seed, _ = WORKLOADS[wid]
    esize = 2 if dtype == "bfloat16" else 4
    block = max(1, (1 << 24) // count)
    native.reducescatter(dtype, n, 1, dist=dist, seed=seed)  # load the library and the table first
    t0 = time.perf_counter()
    used = 0
    for r0 in range(0, n, block):
        out = native.reducescatter(dtype, n, count, dist=dist, seed=seed, r0=r0, r1=min(n, r0 + block),
                                   want=("pat", "sum"))
        used = max(used, out["threads"])
    elapsed = time.perf_counter() - t0
    bus_bytes = float(n) * (n - 1) * count * esize
    return {"value": round(bus_bytes / elapsed / 1e9, 3), "unit": "GB/s", "cores": used, "kind": "oracle",
            "cpu_model": _cpu_model(), "host_cpus_visible": os.cpu_count(),
            "input_gbps": round(float(n) * n * count * esize / elapsed / 1e9, 3),
            "sample": f"whole operation: all {n} destination chunks x all {count} elements, N = {n} inputs each "
                      f"regenerated from the seed; PAT association ({'int32' if dtype == 'int32' else 'float32'}) "
                      f"and fp64 plain sum; C++ std::thread oracle on {used} threads; {elapsed:.1f} s",
            "seconds": round(elapsed, 2)}


def cpu_baseline_ag(wid, min_seconds=1.0):
    """All-gather: the threaded C++ oracle over the whole operation -- every
    receiver's row, the concatenation of the N send buffers regenerated from
    the seed -- on every CPU this process may use, in blocks of receivers that
    keep the host buffer under 256 MiB; repeated until at least `min_seconds`
    have passed (small operations take milliseconds)."""
    import numpy as np

    from oracle import native

    coll, n, count, dtype, dist, seed, _ = WORKLOADS[wid]
    esize = 2 if dtype == "bfloat16" else 4
    block = max(1, (256 << 20) // max(1, n * count * esize))
    np_dtype = {"int32": np.int32, "float32": np.float32, "bfloat16": np.uint16}[dtype]
    buf = np.empty((min(block, n), n * count), dtype=np_dtype)
    native.allgather(dtype, n, 1, dist=dist, seed=seed)  # load the library and the table first
    used, reps = 0, 0
    t0 = time.perf_counter()
    while True:
        # receiver 0's row, from the generator, is the send buffers: the other
        # blocks copy from it instead of generating them again
        row0, used = native.allgather(dtype, n, count, dist=dist, seed=seed, r0=0, r1=1, out=buf[:1])
        inputs = row0.reshape(n, count).copy()
        for r0 in range(1, n, block):
            r1 = min(n, r0 + block)
            _, u = native.allgather(dtype, n, count, inputs=inputs, r0=r0, r1=r1, out=buf[:r1 - r0])
            used = max(used, u)
        reps += 1
        elapsed = time.perf_counter() - t0
        if elapsed >= min_seconds:
            break
    bus_bytes = float(n) * (n - 1) * count * esize * reps
    return {"value": round(bus_bytes / elapsed / 1e9, 3), "unit": "GB/s", "cores": used, "kind": "oracle",
            "cpu_model": _cpu_model(), "host_cpus_visible": os.cpu_count(),
            "sample": f"whole operation x {reps}: all {n} receivers x all {n} chunks of {count} elements, the send "
                      f"buffers regenerated from the seed; concatenation; C++ std::thread oracle on {used} threads; "
                      f"{elapsed:.2f} s",
            "seconds": round(elapsed, 2)}


def small_size_latency(reps=200):
    """The small-size regime: N = 1000 virtual ranks, 64 fp32 (256 B) per chunk,
    U[-1, 1) from seed 0x5041544.  Microseconds per all-gather and per
    reduce-scatter (HIP events around `reps` back-to-back operations), and the
    step count beside log2 N and a ring's N - 1."""
    import math

    import torch

    import synth
    from paper_2506_20252_amd import pat

    n, count, seed = 1000, 64, 0x5041544
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    out = {"workload": "N=1000 virtual ranks, 64 fp32 (256 B) per chunk, U[-1,1)", "log2_n": round(math.log2(n), 3),
           "ring_steps": n - 1}
    for coll in ("allgather", "reducescatter"):
        if coll == "reducescatter":
            send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
            recv = torch.empty((n, count), dtype=torch.float32, device=dev)
        else:
            send = torch.empty((n, count), dtype=torch.float32, device=dev)
            recv = torch.empty((n, n * count), dtype=torch.float32, device=dev)
        for x in range(n):
            synth.fill(send[x], "f32_pm1", seed, x)
        S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))
        if coll == "reducescatter":
            op = lambda: pat.pat_reducescatter(S, R, count, "float32", pat.PAT_SUM, n, stream)  # noqa: E731
            code = pat.PAT_REDUCESCATTER
        else:
            op = lambda: pat.pat_allgather(S, R, count, "float32", n, stream)  # noqa: E731
            code = pat.PAT_ALLGATHER
        for _ in range(5):
            pat.check(op())
        mean_ms, per = time_pair_and_reps(op, stream, reps)
        pat.check(pat.pat_check_device_status(stream))
        st, info = pat.pat_plan_info(code, n, count, "float32")
        out[f"{coll}_us"] = round(mean_ms * 1e3, 2)
        out[f"{coll}_median_us"] = round(statistics.median(per) * 1e3, 2)
        out["steps"] = info["steps"]
        out[f"{coll}_launches"] = info["launches_per_op"]  # the far fusable steps run as one launch
        del send, recv, S, R
    torch.cuda.empty_cache()
    return out


def other_workloads(reps=50):
    """Workloads 1-3 timed the same way (HIP events around back-to-back
    operations): microseconds per operation, aggregate bus bandwidth and the
    fraction of HBM peak that the algorithmic bytes reach.  Last, workload 3
    with one element fewer per chunk: rows that are only element-aligned and
    chunks that end in a partial vector, the relaxed 128-bit kernels' case."""
    import torch

    import synth
    from paper_2506_20252_amd import pat

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    tdt = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}
    rows = []
    for wid, odd in ((1, False), (2, False), (3, False), (3, True)):
        coll, n, count, dtype, dist, seed, desc = WORKLOADS[wid]
        if odd:
            count -= 1
            desc = (f"PAT reduce-scatter (sum), N={n} virtual ranks, fp32 N(0,1), {count}-element output chunk "
                    "(odd count: element-aligned rows, partial last vectors)")
        if coll == "rs":
            send = torch.empty((n, n * count), dtype=tdt[dtype], device=dev)
            recv = torch.empty((n, count), dtype=tdt[dtype], device=dev)
            code = pat.PAT_REDUCESCATTER
        else:
            send = torch.empty((n, count), dtype=tdt[dtype], device=dev)
            recv = torch.empty((n, n * count), dtype=tdt[dtype], device=dev)
            code = pat.PAT_ALLGATHER
        for x in range(n):
            synth.fill(send[x], dist, seed, x)
        S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))

        def op():
            if coll == "rs":
                return pat.pat_reducescatter(S, R, count, dtype, pat.PAT_SUM, n, stream)
            return pat.pat_allgather(S, R, count, dtype, n, stream)

        for _ in range(5):
            pat.check(op())
        mean_ms, per = time_pair_and_reps(op, stream, reps)
        pat.check(pat.pat_check_device_status(stream))
        sec = mean_ms / 1e3
        st, info = pat.pat_plan_info(code, n, count, dtype)
        rows.append({"workload": desc, "us": round(sec * 1e6, 2), "median_us": round(statistics.median(per) * 1e3, 2),
                     "steps": info["steps"],
                     "launches": info["launches_per_op"],
                     "bus_gbps": round(n * info["bus_bytes_per_rank"] / sec / 1e9, 2),
                     "hbm_frac_alg": round(info["alg_bytes"] / sec / 1e9 / HBM_PEAK_GBPS, 4)})
        del send, recv, S, R
    torch.cuda.empty_cache()
    return rows


def streaming_ceiling(nbytes=4 << 30, reps=10):
    """The GPU's streaming bandwidth for the step kernels' access shapes, from
    the plain probe kernels of libpatceiling.so (one 16-byte vector per lane,
    nontemporal): a read-only and a write-only stream, a copy (an all-gather
    step into leaves), a copy into two buffers (an all-gather step into
    forwarding receivers), and a float32 add of two buffers into a third (the
    reduce-scatter shape).  GB/s of bytes read + written."""
    import ctypes

    import torch

    path = os.path.join(ROOT, "paper_2506_20252_amd", "libpatceiling.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    for name, nargs in (("pat_ceiling_copy", 2), ("pat_ceiling_copy2", 3), ("pat_ceiling_add", 3),
                        ("pat_ceiling_read", 2)):
        fn = getattr(lib, name)
        fn.argtypes = [ctypes.c_void_p] * nargs + [ctypes.c_size_t, ctypes.c_void_p]
        fn.restype = ctypes.c_int
    lib.pat_ceiling_write.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint32, ctypes.c_void_p]
    lib.pat_ceiling_write.restype = ctypes.c_int
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    a = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    b = torch.full_like(a, 2.0)
    c = torch.empty_like(a)
    sink = torch.zeros(1024, dtype=torch.int32, device=dev)
    out = {"bytes_per_buffer": nbytes, "kernel": "16 B/lane, 256 lanes/workgroup, nontemporal"}
    # the two-buffer copy runs last: it overwrites b, an input of the add;
    # the write-only stream fills c before the copy overwrites it
    runs = (("read_gbps", 1, lambda: lib.pat_ceiling_read(a.data_ptr(), sink.data_ptr(), nbytes, stream.cuda_stream)),
            ("write_gbps", 1, lambda: lib.pat_ceiling_write(c.data_ptr(), nbytes, 0x40400000, stream.cuda_stream)),
            ("copy_gbps", 2, lambda: lib.pat_ceiling_copy(a.data_ptr(), c.data_ptr(), nbytes, stream.cuda_stream)),
            ("rs_shape_gbps", 3, lambda: lib.pat_ceiling_add(a.data_ptr(), b.data_ptr(), c.data_ptr(), nbytes,
                                                             stream.cuda_stream)),
            ("ag_shape_gbps", 3, lambda: lib.pat_ceiling_copy2(a.data_ptr(), c.data_ptr(), b.data_ptr(), nbytes,
                                                               stream.cuda_stream)))
    for key, streams, op in runs:
        for _ in range(2):
            if op() != 0:
                raise RuntimeError(f"{key}: launch failed")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            op()
        e1.record(stream)
        torch.cuda.synchronize()
        out[key] = round(streams * nbytes * reps / (e0.elapsed_time(e1) / 1e3) / 1e9, 1)
        if key == "rs_shape_gbps" and not bool(torch.equal(c[:1 << 20], torch.full_like(c[:1 << 20], 3.0))):
            raise RuntimeError("ceiling probe: wrong sum")
        if key == "write_gbps" and not bool(torch.equal(c[-(1 << 20):], torch.full_like(c[-(1 << 20):], 3.0))):
            raise RuntimeError("ceiling probe: wrong fill")  # 0x40400000 is float32 3.0
        if key == "read_gbps" and bool(sink.any()):
            raise RuntimeError("ceiling probe: the read found a pattern its input does not hold")
    if not (bool(torch.equal(b[:1 << 20], a[:1 << 20])) and bool(torch.equal(c[:1 << 20], a[:1 << 20]))):
        raise RuntimeError("ceiling probe: wrong two-buffer copy")
    del a, b, c, sink
    torch.cuda.empty_cache()
    return out


def misalign_probe(chunks=500000, reps=20):
    """Why misaligned receive buffers cost the all-gather: 256-byte chunk
    copies (libpatceiling.so) at skew 0 and 4 bytes, all chunks in one launch,
    or even chunks then odd chunks in two launches (lines shared by two chunks
    then written partly in each launch, as the all-gather's steps fill a
    receive buffer).  Microseconds per copy of every chunk."""
    import ctypes

    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2506_20252_amd", "libpatceiling.so"))
    fn = lib.pat_ceiling_chunk_copy
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    n = chunks * 256 + 256
    src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    dst = torch.zeros(n, dtype=torch.uint8, device="cuda:0")
    stream = torch.cuda.current_stream()
    rows = []
    for skew in (0, 4):
        for split in (False, True):
            def op():
                for par in ((0, 1) if split else (-1,)):
                    if fn(src.data_ptr(), dst.data_ptr(), chunks, skew, par, stream.cuda_stream) != 0:
                        raise RuntimeError("chunk copy probe: launch failed")
            op()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                op()
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            rows.append({"skew_bytes": skew, "launches": 2 if split else 1, "us": round(us, 2),
                         "gbps_read_plus_write": round(2 * chunks * 256 / (us * 1e-6) / 1e9, 1)})
    if not bool(torch.equal(dst[4:4 + chunks * 256], src[4:4 + chunks * 256])):
        raise RuntimeError("chunk copy probe: wrong copy")
    del src, dst
    torch.cuda.empty_cache()
    print(json.dumps({"metric": "256-byte chunk copies at a skew (why misaligned all-gathers cost more)",
                      "chunks": chunks, "rows": rows, "allgather": misaligned_allgather()}), flush=True)


def misaligned_allgather(n=1000, reps=50):
    """The all-gather of workload 6's shape (N=1000, float32) with every row
    16-byte aligned (64 elements), every row one element off a 16-byte
    boundary (64 elements), and an odd count (63 elements): microseconds per
    operation (median of 5 runs of `reps`), each result checked on 4 rows."""
    import torch

    import synth
    from paper_2506_20252_amd import pat

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    out = []
    for label, count, skew in (("aligned", 64, 0), ("one element off", 64, 1), ("odd count", 63, 0)):
        sstride, rstride = count + skew, n * count + skew
        sflat = torch.empty(n * sstride + skew, dtype=torch.float32, device=dev)
        rflat = torch.empty(n * rstride + skew, dtype=torch.float32, device=dev)
        send = [sflat[skew + r * sstride: skew + r * sstride + count] for r in range(n)]
        recv = [rflat[skew + r * rstride: skew + r * rstride + n * count] for r in range(n)]
        for x in range(n):
            synth.fill(send[x], "f32_pm1", 0x5041544, x)
        S, R = pat.pointer_array(send), pat.pointer_array(recv)
        for _ in range(3):
            pat.check(pat.pat_allgather(S, R, count, "float32", n, stream))
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(reps):
                pat.check(pat.pat_allgather(S, R, count, "float32", n, stream))
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3 / reps)
        host = torch.stack([x.cpu() for x in send])
        if not all(torch.equal(recv[r].cpu().view(n, count), host) for r in (0, 1, n // 2, n - 1)):
            raise RuntimeError(f"misaligned all-gather probe ({label}): wrong result")
        out.append({"case": label, "count": count, "row_offset_elems": skew, "us": round(statistics.median(ts), 1)})
        del send, recv, S, R, sflat, rflat
        torch.cuda.empty_cache()
    return out


def budget_sweep(wid, reps, max_slot_bytes=32 << 30, aggregation="pow2"):
    """Time one workload at every aggregation level: the budget is set to the
    bytes of the largest step at T = 1, 2, 4, ... up to full aggregation, so
    the plan goes from one linear tree (N - 1 steps) to ceil(log2 N) steps,
    stopping early once the slots of all ranks would exceed max_slot_bytes.
    With aggregation "budget" the budget also takes 3, 5, 6 and 7 chunks
    (K chunks per step, the list schedule where it is shorter)."""
    import torch

    import synth
    from paper_2506_20252_amd import pat

    coll, n, count, dtype, dist, seed, desc = WORKLOADS[wid]
    tdt = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}[dtype]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    if coll == "rs":
        send = torch.empty((n, n * count), dtype=tdt, device=dev)
        recv = torch.empty((n, count), dtype=tdt, device=dev)
        code = pat.PAT_REDUCESCATTER
    else:
        send = torch.empty((n, count), dtype=tdt, device=dev)
        recv = torch.empty((n, n * count), dtype=tdt, device=dev)
        code = pat.PAT_ALLGATHER
    for x in range(n):
        synth.fill(send[x], dist, seed, x)
    S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))
    slot_elem = 4 if (coll == "rs" or dtype != "bfloat16") else (2 if dtype == "bfloat16" else 4)
    pat.check(pat.pat_set_aggregation(aggregation))
    rows = []
    Ks = [1, 2, 3, 4, 5, 6, 7, 8] if aggregation == "budget" else []
    T = 1
    while True:
        if Ks:
            T = Ks.pop(0)
        budget = T * count * slot_elem
        pat.check(pat.pat_set_buffer_bytes(budget))
        st, info = pat.pat_plan_info(code, n, count, dtype)
        if (info["T"] < T and not info["list_schedule"]) or info["slot_bytes_total"] > max_slot_bytes:
            if Ks:
                continue
            break

        def op():
            if coll == "rs":
                return pat.pat_reducescatter(S, R, count, dtype, pat.PAT_SUM, n, stream)
            return pat.pat_allgather(S, R, count, dtype, n, stream)

        for _ in range(3):
            pat.check(op())
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            pat.check(op())
        e1.record(stream)
        torch.cuda.synchronize()
        pat.check(pat.pat_check_device_status(stream))
        sec = e0.elapsed_time(e1) / 1e3 / reps
        rows.append({"budget_bytes": budget, "T": info["T"], "list_schedule": bool(info["list_schedule"]),
                     "steps": info["steps"],
                     "launches": info["launches_per_op"],
                     "slot_bytes_per_rank": info["slot_bytes_per_rank"], "us": round(sec * 1e6, 2),
                     "bus_gbps": round(n * info["bus_bytes_per_rank"] / sec / 1e9, 2),
                     "hbm_frac_alg": round(info["alg_bytes"] / sec / 1e9 / HBM_PEAK_GBPS, 4)})
        pat.check(pat.pat_finalize())
        if Ks:
            continue
        if info["T"] * 2 > (1 << max(info["L"] - 1, 0)):
            break
        T *= 2  # after the listed K (1 .. 8 with "budget"), powers of two
    pat.check(pat.pat_set_buffer_bytes(0))
    pat.check(pat.pat_set_aggregation("pow2"))
    print(json.dumps({"metric": "PAT budget sweep (steps and time per aggregation level)", "workload": desc,
                      "aggregation": aggregation, "exec_mode": ["persistent", "graph", "stream", "dataflow"][pat.pat_get_exec_mode()],
                      "nranks": n, "log2_n": round(math.log2(n), 3), "rows": rows}), flush=True)


def size_sweep(n=128, max_input_bytes=16 << 30, reps_bytes=32 << 30):
    """Both collectives at one rank count over chunk sizes from 256 B up, at
    the default budget: microseconds per operation, steps and launches, bus
    bandwidth and the fraction of HBM peak that the algorithmic bytes reach --
    where the latency regime ends and the bandwidth roofline begins.  float32
    reduce-scatter and all-gather, N(0,1) inputs, seed 0x5153."""
    import torch

    import synth
    from paper_2506_20252_amd import pat

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    rows = []
    for coll in ("rs", "ag"):
        count = 64  # 256 B
        while n * n * count * 4 <= max_input_bytes:
            if coll == "rs":
                send = torch.empty((n, n * count), dtype=torch.float32, device=dev)
                recv = torch.empty((n, count), dtype=torch.float32, device=dev)
                code = pat.PAT_REDUCESCATTER
            else:
                send = torch.empty((n, count), dtype=torch.float32, device=dev)
                recv = torch.empty((n, n * count), dtype=torch.float32, device=dev)
                code = pat.PAT_ALLGATHER
            for x in range(n):
                synth.fill(send[x], "f32_normal", 0x5153, x)
            S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))

            def op():
                if coll == "rs":
                    return pat.pat_reducescatter(S, R, count, "float32", pat.PAT_SUM, n, stream)
                return pat.pat_allgather(S, R, count, "float32", n, stream)

            st, info = pat.pat_plan_info(code, n, count, "float32")
            reps = int(max(5, min(200, reps_bytes / max(info["alg_bytes"], 1.0))))
            for _ in range(3):
                pat.check(op())
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(reps):
                pat.check(op())
            e1.record(stream)
            torch.cuda.synchronize()
            pat.check(pat.pat_check_device_status(stream))
            sec = e0.elapsed_time(e1) / 1e3 / reps
            rows.append({"collective": "reduce-scatter" if coll == "rs" else "all-gather", "chunk_bytes": count * 4,
                         "T": info["T"], "steps": info["steps"], "launches": info["launches_per_op"],
                         "streaming": bool(info["streaming"]), "us": round(sec * 1e6, 2),
                         "bus_gbps": round(n * info["bus_bytes_per_rank"] / sec / 1e9, 1),
                         "hbm_frac_alg": round(info["alg_bytes"] / sec / 1e9 / HBM_PEAK_GBPS, 4)})
            print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
            del send, recv, S, R
            pat.check(pat.pat_finalize())
            torch.cuda.empty_cache()
            count *= 4
    print(json.dumps({"metric": "PAT size sweep (float32, default budget, stream mode)", "nranks": n,
                      "rows": rows}), flush=True)


def copy_probe(nbytes, reps, kind="torch"):
    """A plain device-to-device copy of known size: reads and writes nbytes.
    kind "torch": torch's copy (the runtime's __amd_rocclr_copyBuffer);
    kind "nt": the nontemporal 16-byte-per-lane copy of libpatceiling.so, the
    access type of the step kernels on large operations."""
    import ctypes

    import torch
    n = nbytes // 2
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda:0")
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream()
    if kind == "nt":
        lib = ctypes.CDLL(os.path.join(ROOT, "paper_2506_20252_amd", "libpatceiling.so"))
        lib.pat_ceiling_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        lib.pat_ceiling_copy.restype = ctypes.c_int

        def op():
            if lib.pat_ceiling_copy(src.data_ptr(), dst.data_ptr(), 2 * n, stream.cuda_stream) != 0:
                raise RuntimeError("copy probe launch failed")
    else:
        def op():
            dst.copy_(src)
    op()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        op()
    e1.record(stream)
    torch.cuda.synchronize()
    if not bool(torch.equal(dst[:1 << 20], src[:1 << 20])):
        raise RuntimeError("copy probe: wrong copy")
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"kind": kind, "copy_bytes": 2 * n, "read_bytes": 2 * n, "write_bytes": 2 * n,
                      "ms": round(ms, 4), "GBps_read_plus_write": round(4 * n / ms / 1e6, 1)}), flush=True)


def time_ops(op, stream, reps):
    """Runs `op` reps times back to back on `stream` with a HIP event recorded
    before the first and after each one.  Returns (mean ms per operation over
    the whole run, list of per-operation ms)."""
    import torch

    from paper_2506_20252_amd import pat
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k in range(reps):
        pat.check(op(), "timed")
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    per = [evs[k].elapsed_time(evs[k + 1]) for k in range(reps)]
    return evs[0].elapsed_time(evs[-1]) / reps, per


def time_pair_and_reps(op, stream, reps):
    """For short operations: the mean over `reps` back-to-back operations
    under one event pair (no events between them), then a second run of
    `reps` with an event after each one for the per-operation times."""
    import torch

    from paper_2506_20252_amd import pat
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        pat.check(op())
    e1.record(stream)
    torch.cuda.synchronize()
    _, per = time_ops(op, stream, reps)
    return e0.elapsed_time(e1) / reps, per


def kernel_name(coll, dtype, path, streaming, kind):
    """The kernel template a launch runs (as rocprofv3 names it, abridged)."""
    if coll == "rs":
        traits = {"int32": "TI32", "float32": "TF32", "bfloat16": "TB16"}[dtype] + {0: "S", 1: "V", 2: "U"}[path]
        op = f"RsOp<{traits}, {'true' if streaming else 'false'}>"
    else:
        op = {0: "AgOp<element>", 1: "AgOp<v4u>", 2: "AgOp<v4u, relaxed>"}[path]
        op = op[:-1] + f", nontemporal={'true' if streaming else 'false'}>"
    return ("tree_kernel<" if kind == 1 else "step_kernel<") + op + ">"


def kernel_roofline(info, coll, dtype, reps):
    """The launch trace of the first `reps` timed operations: a HIP event pair
    around every kernel launch, recorded by the library on the kernels' stream
    (armed before the timed region), and each launch's algorithmic bytes from
    the plan's byte model.  The dominant kernel is the one with the most traced
    time; its rate is its launches' bytes over their summed durations."""
    from paper_2506_20252_amd import pat
    launches = info["launches_per_op"]
    st, rows = pat.pat_trace_read(reps * launches)
    pat.check(st, "pat_trace_read")
    if len(rows) != reps * launches:
        raise RuntimeError(f"trace: {len(rows)} launches recorded, {reps * launches} expected")
    by = {}
    for ms, nbytes, kind, _step in rows:
        g = by.setdefault(kind, {"ms": 0.0, "bytes": 0.0, "launches": 0, "rates": []})
        g["ms"] += ms
        g["bytes"] += nbytes
        g["launches"] += 1
        g["rates"].append(nbytes / (ms / 1e3) / 1e9 if ms > 0 else 0.0)
    op_bytes = sum(r[1] for r in rows) / reps
    if abs(op_bytes - info["alg_bytes"]) > 1e-6 * info["alg_bytes"]:
        raise RuntimeError(f"trace bytes per operation {op_bytes} != plan {info['alg_bytes']}")
    dom = max(by, key=lambda k: by[k]["ms"])
    g = by[dom]
    achieved = g["bytes"] / (g["ms"] / 1e3) / 1e9
    rates = sorted(g["rates"])
    kinds = [{"kernel": kernel_name(coll, dtype, info["vector_path"], info["streaming"], k),
              "launches_per_op": v["launches"] // reps, "bytes_per_launch": round(v["bytes"] / v["launches"], 1),
              "avg_launch_us": round(v["ms"] / v["launches"] * 1e3, 3),
              "frac": round(v["bytes"] / (v["ms"] / 1e3) / 1e9 / HBM_PEAK_GBPS, 4)} for k, v in sorted(by.items())]
    return {
        "kernel": kernel_name(coll, dtype, info["vector_path"], info["streaming"], dom),
        "achieved": achieved,
        "launches_per_op": g["launches"] // reps,
        "avg_launch_us": round(g["ms"] / g["launches"] * 1e3, 3),
        "bytes_per_launch": round(g["bytes"] / g["launches"], 1),
        "share_of_traced_time": round(g["ms"] / sum(v["ms"] for v in by.values()), 4),
        "launch_frac": {"min": round(rates[0] / HBM_PEAK_GBPS, 4),
                        "median": round(statistics.median(rates) / HBM_PEAK_GBPS, 4),
                        "max": round(rates[-1] / HBM_PEAK_GBPS, 4)},
        "traced_ops": reps,
        "timing": f"HIP event pair around each launch of the first {reps} timed operations, on the kernels' "
                  "stream (library launch trace)",
        "kernels": kinds,
    }


def step_clock_report(wid, reps=5):
    """The fused launch of one workload, step by step: with PAT_STEP_CLOCK=1
    the fused kernel records the device wall clock per workgroup before its
    first step and after each one.  Reports, per fused step, its distance,
    chunks per rank, algorithmic bytes and the median / 90th percentile over
    workgroups of its duration, and the launch's first-to-last stamp span
    (the last of `reps` operations)."""
    import numpy as np
    import torch

    import synth
    from paper_2506_20252_amd import pat

    coll, n, count, dtype, dist, seed, desc = WORKLOADS[wid]
    tdt = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}[dtype]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    pat.check(pat.pat_set_exec_mode("stream"))
    if coll == "rs":
        send, recv = torch.empty((n, n * count), dtype=tdt, device=dev), torch.empty((n, count), dtype=tdt, device=dev)
        code = pat.PAT_REDUCESCATTER
    else:
        send, recv = torch.empty((n, count), dtype=tdt, device=dev), torch.empty((n, n * count), dtype=tdt, device=dev)
        code = pat.PAT_ALLGATHER
    for x in range(n):
        synth.fill(send[x], dist, seed, x)
    S, R = pat.pointer_array(list(send)), pat.pointer_array(list(recv))

    def op():
        if coll == "rs":
            return pat.pat_reducescatter(S, R, count, dtype, pat.PAT_SUM, n, stream)
        return pat.pat_allgather(S, R, count, dtype, n, stream)

    st, info = pat.pat_plan_info(code, n, count, dtype)
    pat.check(pat.pat_trace_start(reps * info["launches_per_op"]))
    for _ in range(reps):
        pat.check(op())
    torch.cuda.synchronize()
    st, launches = pat.pat_trace_read(reps * info["launches_per_op"])
    pat.check(st)
    st, stamps, tpu = pat.pat_step_clock(code, n, count, dtype)
    pat.check(st, "pat_step_clock")
    st, steps, entries = pat.pat_plan_steps(code, n, count, dtype)
    fused = [r for r in launches[-info["launches_per_op"]:] if r[2] == 1]
    s0 = fused[0][3] if fused else 0
    dur = np.diff(stamps.astype(np.int64), axis=1) / tpu
    rows = []
    for k in range(dur.shape[1]):
        d, kk = steps[s0 + k]
        rows.append({"step": s0 + k, "distance": d, "chunks_per_rank": kk,
                     "median_us": round(float(np.median(dur[:, k])), 3),
                     "p90_us": round(float(np.percentile(dur[:, k], 90)), 3)})
    print(json.dumps({"metric": "PAT fused launch, per-step device clock (median over workgroups)",
                      "workload": desc, "workgroups": int(stamps.shape[0]), "fused_steps": dur.shape[1],
                      "launch_us_event": round(fused[-1][0] * 1e3, 3) if fused else None,
                      "launch_bytes": fused[-1][1] if fused else None,
                      "span_us": round(float((stamps[:, -1].max() - stamps[:, 0].min()) / tpu), 3),
                      "first_stamp_spread_us": round(float((stamps[:, 0].max() - stamps[:, 0].min()) / tpu), 3),
                      "steps": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--mode", default="stream", choices=["persistent", "graph", "stream", "dataflow"])
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="instead: time a plain device copy of BYTES (the achievable-bandwidth line, and "
                         "the calibration kernel for the memory-traffic counters)")
    ap.add_argument("--copy-probe-kind", default="torch", choices=["torch", "nt"])
    ap.add_argument("--workload", type=int, default=5, choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=1.0,
                    help="all-gather CPU baseline: repeat the whole operation for at least this long")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-latency", action="store_true", help="skip the small-size latency figures")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the streaming-ceiling probes")
    ap.add_argument("--budget-sweep", action="store_true",
                    help="instead: time the workload at every aggregation level (T = 1 .. full)")
    ap.add_argument("--aggregation", default="pow2", choices=["pow2", "budget"],
                    help="with --budget-sweep: power-of-two sub-trees, or any chunks per step (list schedule)")
    ap.add_argument("--misalign-probe", action="store_true",
                    help="instead: 256-byte chunk copies at a skew, one launch or even/odd chunks in two, and "
                         "the N=1000 all-gather aligned, one element off and with an odd count")
    ap.add_argument("--step-clock", action="store_true",
                    help="instead: per-step device clock of the workload's fused launch (PAT_STEP_CLOCK=1)")
    ap.add_argument("--size-sweep", action="store_true",
                    help="instead: both collectives at N=128 over chunk sizes from 256 B (float32)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: all virtual ranks are emulated on one GPU; runs on more than one GPU "
              "are not supported (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_probe:
        copy_probe(args.copy_probe, args.steps, args.copy_probe_kind)
        return
    from paper_2506_20252_amd import pat as _pat
    _pat.check(_pat.pat_set_exec_mode(args.mode))  # the sweeps run in the chosen mode too
    if args.budget_sweep:
        budget_sweep(args.workload, args.steps, aggregation=args.aggregation)
        return
    if args.size_sweep:
        size_sweep()
        return
    if args.misalign_probe:
        misalign_probe()
        return
    if args.step_clock:
        os.environ["PAT_STEP_CLOCK"] = "1"  # read when the plan is made
        step_clock_report(args.workload)
        return

    import synth
    from paper_2506_20252_amd import pat

    coll, n, count, dtype, dist, seed, desc = WORKLOADS[args.workload]
    tdt = {"int32": torch.int32, "float32": torch.float32, "bfloat16": torch.bfloat16}[dtype]
    esize = 2 if dtype == "bfloat16" else 4
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    pat.lib()
    pat.check(pat.pat_set_exec_mode(args.mode))

    if coll == "rs":
        send = torch.empty((n, n * count), dtype=tdt, device=dev)
        recv = torch.empty((n, count), dtype=tdt, device=dev)
        code = pat.PAT_REDUCESCATTER
    else:
        send = torch.empty((n, count), dtype=tdt, device=dev)
        recv = torch.empty((n, n * count), dtype=tdt, device=dev)
        code = pat.PAT_ALLGATHER
    for x in range(n):
        synth.fill(send[x], dist, seed, x)
    # Pointer arrays built once: the timed calls pass them straight to the C-ABI.
    sends, recvs = pat.pointer_array(list(send)), pat.pointer_array(list(recv))
    torch.cuda.synchronize()

    st, info = pat.pat_plan_info(code, n, count, dtype)
    pat.check(st)

    def op():
        if coll == "rs":
            return pat.pat_reducescatter(sends, recvs, count, dtype, pat.PAT_SUM, n, stream)
        return pat.pat_allgather(sends, recvs, count, dtype, n, stream)

    for _ in range(args.warmup):
        pat.check(op(), "warmup")
    torch.cuda.synchronize()
    pat.check(pat.pat_check_device_status(stream))

    # The launch trace covers the first operations of the timed region: an
    # event pair around each launch adds a few microseconds per launch, so
    # tracing all of them would slow the timed operations measurably (1% on
    # workload 5, 16% on workload 4); three traced operations of twenty cost
    # the mean under 0.2% on workload 5.
    traced = min(args.steps, 3, (1 << 20) // max(1, info["launches_per_op"]))
    if args.mode == "stream":
        pat.check(pat.pat_trace_start(traced * info["launches_per_op"]))
    ms, rep_ms = time_ops(op, stream, args.steps)
    pat.check(pat.pat_check_device_status(stream))
    sec = ms / 1e3
    bus_per_rank = info["bus_bytes_per_rank"]
    if args.mode == "stream":
        roof = kernel_roofline(info, coll, dtype, traced)
    else:
        # no per-launch trace in these modes: the operation's time spread over its launches
        launches = 1 if args.mode == "persistent" else info["launches_per_op"]
        roof = {"kernel": "persistent_kernel" if args.mode == "persistent" else "step_kernel",
                "achieved": info["alg_bytes"] / launches / (sec / launches) / 1e9, "launches_per_op": launches,
                "timing": "operation time / launches (no per-launch trace in this mode)"}
    achieved = roof.pop("achieved")
    traffic = committed_traffic(args.workload, args.mode, roof["kernel"])
    if traffic is not None and roof.get("avg_launch_us"):
        # the counted HBM-side bytes over the same launch time: how busy HBM
        # itself was (below `frac` where the kernel hits in cache)
        roof["traffic_frac"] = round(traffic / (roof["avg_launch_us"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)

    out = {
        "metric": METRIC,
        "value": round(n * bus_per_rank / sec / 1e9, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "median_ms_per_step": round(statistics.median(rep_ms), 4),
        "rep_ms": {"min": round(min(rep_ms), 4), "max": round(max(rep_ms), 4), "reps": len(rep_ms)},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if coll == "rs" and dtype != "int32" else ("int32" if dtype == "int32" else "bytes"),
        "data": "synthetic",
        "config": {"workload": desc, "nranks": n, "count": count, "input_dtype": dtype,
                   "collective": "reduce-scatter" if coll == "rs" else "all-gather", "exec_mode": args.mode,
                   "buffer_bytes_per_slot": pat.pat_get_buffer_bytes(), "T": info["T"],
                   "pat_steps": info["steps"], "pieces": info["pieces"],
                   "fused_steps": 0 if args.mode == "persistent" else info["fused_steps"],
                   "streaming_accesses": bool(info["streaming"]), "xcd_run": info["xcd_run"],
                   "seed": seed},
        "bus_gbps_per_rank": round(bus_per_rank / sec / 1e9, 4),
        "latency_us": round(ms * 1e3, 2),
        "alg_bytes_per_op": info["alg_bytes"],
        "hbm_frac_alg": round(info["alg_bytes"] / sec / 1e9 / HBM_PEAK_GBPS, 4),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic, **roof},
    }
    if not args.no_latency:
        out["small_size_latency"] = small_size_latency()
        out["other_workloads"] = other_workloads()
    if not args.no_cpu_baseline:
        if coll == "rs":
            out["cpu_baseline"] = cpu_baseline_rs(args.workload)
        else:
            out["cpu_baseline"] = cpu_baseline_ag(args.workload, args.cpu_seconds)
    del send, recv, sends, recvs
    torch.cuda.empty_cache()
    if not args.no_ceiling:
        ceil = streaming_ceiling()
        shape_key = "rs_shape_gbps" if coll == "rs" else "ag_shape_gbps"
        ceil["roofline_achieved_over_" + shape_key] = round(achieved / ceil[shape_key], 4)
        out["streaming_ceiling"] = ceil
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
