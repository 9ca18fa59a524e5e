"""Pins for the threaded C++ oracle (oracle/rs_oracle.cpp, oracle/ag_oracle.cpp):
it must agree with the Python oracle, which the pins in test_oracle_pins.py tie
to the paper.

* PAT association: bit-exact against the step-by-step executor
  (oracle.pat.reducescatter, a different construction: explicit steps and
  buffers) for N <= 64, every aggregation level, float32 and bfloat16;
* int32: equal to the definition (integer adds associate);
* the fp64 plain sum and absolute sum: equal to oracle.definitions;
* regenerated inputs: equal to the array path fed with the host twin of the
  generator;
* results do not depend on the thread count or on the destination range;
* bf16 rounding ties go to even;
* all-gather: every receiver's row is the concatenation of the send buffers
  (oracle.definitions.allgather, and the Bruck / PAT step executors through
  it), from arrays and from regenerated inputs, for any receiver range and
  thread count.
Nothing here calls the HIP library.
"""

import numpy as np
import pytest

import synth
from oracle import definitions as D
from oracle import native
from oracle import pat

RNG = np.random.default_rng(0x0AC1E)


def bf16(shape):
    return D.f32_to_bf16_bits(RNG.standard_normal(shape).astype(np.float32))


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6, 7, 8, 9, 13, 24, 33, 64])
@pytest.mark.parametrize("dtype", ["float32", "bfloat16"])
def test_pat_order_equals_step_executor_every_level(n, dtype):
    m = 5 if n > 24 else 9
    x = RNG.standard_normal((n, n, m)).astype(np.float32) if dtype == "float32" else bf16((n, n, m))
    got = native.reducescatter(dtype, n, m, inputs=x, want=("pat",))["pat"]
    width = np.uint32 if dtype == "float32" else np.uint16
    for t in range(max(pat.ceil_log2(n), 1)):
        ref, _ = pat.reducescatter(x, t, dtype)
        assert (got.view(width) == ref.view(width)).all(), f"t={t}"


@pytest.mark.parametrize("n", [1, 2, 6, 24, 100, 257])
def test_int32_is_the_definition(n):
    x = RNG.integers(-2**31, 2**31, size=(n, n, 7), dtype=np.int64).astype(np.int32)
    out = native.reducescatter("int32", n, 7, inputs=x)
    assert (out["pat"] == D.reducescatter_sum(x, "int32")).all()
    exact = np.stack([x[:, R].astype(np.int64).sum(axis=0) for R in range(n)])
    assert (out["sum"] == exact.astype(np.float64)).all()


@pytest.mark.parametrize("n,dtype", [(6, "float32"), (33, "float32"), (24, "bfloat16"), (128, "bfloat16")])
def test_plain_and_absolute_sums_are_the_definition(n, dtype):
    m = 11
    x = RNG.standard_normal((n, n, m)).astype(np.float32) if dtype == "float32" else bf16((n, n, m))
    out = native.reducescatter(dtype, n, m, inputs=x)
    assert (out["sum"] == D.reducescatter_sum(x, dtype)).all()  # same order: rank 0 .. N-1
    assert (out["abs"] == D.reducescatter_abs_sum(x, dtype)).all()


@pytest.mark.parametrize("dist,dtype", [("int32_pm2p20", "int32"), ("f32_pm1", "float32"),
                                        ("f32_normal", "float32"), ("bf16_normal", "bfloat16")])
def test_regenerated_inputs_equal_the_array_path(dist, dtype):
    n, count, seed = 9, 300, 0x5EED
    host = np.stack([synth.host_buffer(dist, seed, x, n * count) for x in range(n)]).reshape(n, n, count)
    a = native.reducescatter(dtype, n, count, inputs=host)
    g = native.reducescatter(dtype, n, count, dist=dist, seed=seed)
    for k in ("pat", "sum", "abs"):
        assert (a[k] == g[k]).all(), k


def test_threads_and_destination_ranges_do_not_change_results():
    n, count, seed = 37, 5000, 0x7A11
    full = native.reducescatter("float32", n, count, dist="f32_normal", seed=seed, nthreads=0)
    one = native.reducescatter("float32", n, count, dist="f32_normal", seed=seed, nthreads=1)
    assert one["threads"] == 1
    part = native.reducescatter("float32", n, count, dist="f32_normal", seed=seed, r0=5, r1=12, nthreads=3)
    for k in ("pat", "sum", "abs"):
        assert (full[k].view(np.uint64 if k != "pat" else np.uint32) ==
                one[k].view(np.uint64 if k != "pat" else np.uint32)).all()
        assert (part[k] == full[k][5:12]).all()


def test_bf16_rounding_ties_go_to_even():
    # 1 + 2^-8 lies halfway between bf16 1.0 and 1.0078125: even is 1.0.
    # 1.0078125 + 2^-8 lies halfway between 1.0078125 and 1.015625: even is 1.015625.
    x = np.zeros((2, 2, 2), dtype=np.uint16)
    x[0, :, 0], x[1, :, 0] = 0x3F80, 0x3B80      # 1.0 and 2^-8
    x[0, :, 1], x[1, :, 1] = 0x3F81, 0x3B80      # 1.0078125 and 2^-8
    got = native.reducescatter("bfloat16", 2, 2, inputs=x)["pat"]
    assert (got[:, 0] == 0x3F80).all() and (got[:, 1] == 0x3F82).all()


def test_invalid_arguments_are_refused():
    with pytest.raises(ValueError):
        native.reducescatter("float32", 4, 3, inputs=np.zeros((4, 4, 2), np.float32))
    with pytest.raises(ValueError):
        native.reducescatter("float32", 4, 3, dist="f32_normal", r0=2, r1=9)


@pytest.mark.parametrize("dist,dtype", [("int32_pm2p20", "int32"), ("f32_normal", "float32"),
                                        ("bf16_normal", "bfloat16")])
@pytest.mark.parametrize("n,count", [(1, 5), (2, 1), (7, 13), (24, 33), (100, 3)])
def test_allgather_is_the_definition(n, count, dist, dtype):
    seed = 0xA6 + n
    host = np.stack([synth.host_buffer(dist, seed, x, count) for x in range(n)])
    exp = D.allgather(host).reshape(n, n * count)
    got, _ = native.allgather(dtype, n, count, dist=dist, seed=seed)
    assert (got == exp).all()
    arr, _ = native.allgather(dtype, n, count, inputs=host)
    assert (arr == exp).all()
    # and the step executors of the schedule reach the same rows
    ex, _ = pat.allgather(host, max(pat.ceil_log2(n) - 1, 0))
    assert (np.asarray(ex).reshape(n, n * count) == exp).all()


def test_allgather_ranges_threads_and_zero_count():
    n, count, seed = 33, 1000, 0xA6A6
    full, used = native.allgather("float32", n, count, dist="f32_normal", seed=seed)
    assert used >= 1
    one, used1 = native.allgather("float32", n, count, dist="f32_normal", seed=seed, nthreads=1)
    assert used1 == 1 and (one.view(np.uint32) == full.view(np.uint32)).all()
    buf = np.empty((7, n * count), dtype=np.float32)
    part, _ = native.allgather("float32", n, count, dist="f32_normal", seed=seed, r0=20, r1=27, nthreads=3, out=buf)
    assert part is buf and (part.view(np.uint32) == full[20:27].view(np.uint32)).all()
    empty, _ = native.allgather("bfloat16", 5, 0, dist="bf16_normal", seed=1)
    assert empty.shape == (5, 0)
    with pytest.raises(ValueError):
        native.allgather("float32", 4, 3, inputs=np.zeros((4, 2), np.float32))
    with pytest.raises(ValueError):
        native.allgather("float32", 4, 3, dist="f32_normal", r0=2, r1=9)
