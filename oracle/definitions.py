"""What all-gather and reduce-scatter compute, by definition.

Test infrastructure only (see the package docstring).

The paper (section "All-gather and reduce-scatter algorithms") takes the two
operations with MPI semantics: the send buffer is read-only, the all-gather
receive buffer holds the data of every rank, and the reduce-scatter receive
buffer holds one rank's share of the reduction.  Written out:

* all-gather:      out[r][x][i] = in[x][i]              for every rank r
* reduce-scatter:  out[R][i]    = sum over x of in[x][R][i]

Array conventions used throughout the oracle:

* all-gather input  ``(N, m)``      -- rank x sends row x
* all-gather output ``(N, N, m)``   -- [receiving rank, chunk, element]
* reduce-scatter input  ``(N, N, m)`` -- [sending rank, chunk, element]
* reduce-scatter output ``(N, m)``    -- [rank, element]

``m`` is the per-chunk element count (``count``), or the number of sampled
element positions when only a sample of every chunk is checked: both
operations act on each element position independently.

bf16 values are carried as ``uint16`` bit patterns (numpy has no bf16 type).
"""

import numpy as np
import torch


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening: a bf16 value is the upper half of the fp32 with the same
    sign, exponent and leading mantissa bits."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16, round-to-nearest-even, via PyTorch's CPU cast."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def allgather(inputs: np.ndarray) -> np.ndarray:
    """out[r][x] = in[x] for every receiving rank r (a byte copy: any dtype)."""
    inputs = np.asarray(inputs)
    n = inputs.shape[0]
    out = np.empty((n,) + inputs.shape, dtype=inputs.dtype)
    for r in range(n):
        for x in range(n):
            out[r, x] = inputs[x]
    return out


def reducescatter_sum(inputs: np.ndarray, dtype: str) -> np.ndarray:
    """Plain sum over sending ranks, in rank order, in a wide type.

    int32:     exact sum in int64, then wrapped modulo 2**32 (what a two's
               complement int32 accumulation gives in any order).
    float32:   sum in fp64, returned in fp64 (the tolerance reference).
    bfloat16:  inputs widened exactly, summed in fp64, returned in fp64.
    """
    inputs = np.asarray(inputs)
    n = inputs.shape[0]
    if dtype == "int32":
        acc = np.zeros(inputs.shape[2:], dtype=np.int64)
        out = np.empty((n,) + inputs.shape[2:], dtype=np.int32)
        for R in range(n):
            acc[...] = 0
            for x in range(n):
                acc += inputs[x, R].astype(np.int64)
            out[R] = (acc & 0xFFFFFFFF).astype(np.uint32).view(np.int32)
        return out
    if dtype == "float32":
        vals = inputs.astype(np.float64)
    elif dtype == "bfloat16":
        vals = bf16_bits_to_f32(inputs).astype(np.float64)
    else:
        raise ValueError(dtype)
    out = np.zeros((n,) + inputs.shape[2:], dtype=np.float64)
    for R in range(n):
        for x in range(n):
            out[R] += vals[x, R]
    return out


def reducescatter_abs_sum(inputs: np.ndarray, dtype: str) -> np.ndarray:
    """sum over x of |in[x][R][i]| in fp64: the scale of the tolerance test."""
    inputs = np.asarray(inputs)
    if dtype == "float32":
        vals = np.abs(inputs.astype(np.float64))
    elif dtype == "bfloat16":
        vals = np.abs(bf16_bits_to_f32(inputs).astype(np.float64))
    else:
        raise ValueError(dtype)
    n = inputs.shape[0]
    out = np.zeros((n,) + inputs.shape[2:], dtype=np.float64)
    for R in range(n):
        for x in range(n):
            out[R] += vals[x, R]
    return out
