"""Pins for the CPU oracle: checks against what the paper and the mathematics fix.

Nothing here calls the HIP library.  The oracle is checked against
* values the paper prints for its worked examples (tests/golden/*.txt),
* an independent executor of the paper's enumerated Bruck description,
* closed forms written here from the tree definition (not from the oracle),
* invariants the paper states (exactly-once delivery, logarithmic steps for
  small sizes, logarithmic buffers independent of size),
* brute force on tiny rank counts, and
* a rounding-error bound for the float32 accumulation order.
The last block plants plausible mistakes in the oracle and checks that one of
these pins fails.
"""

import math

import numpy as np
import pytest

from conftest import read_golden
from oracle import bruck, pat
from oracle import definitions as D

RNG = np.random.default_rng(20250625)


def full_t(n):
    return max(pat.ceil_log2(n) - 1, 0)


# --------------------------------------------------------------------------
# Section "Binomial-tree based algorithms": Bruck, farthest first, truncation
# --------------------------------------------------------------------------

def test_bruck_steps_match_paper_description():
    g = read_golden("bruck_n8_steps.txt")
    held, log = bruck.allgather(list(range(8)))
    assert [d for d, _ in log] == [1, 2, 4]
    for d, sent in log:
        offsets = [int(x) for x in g[str(d)]]
        for r in range(8):
            assert sent[r] == [(r + o) % 8 for o in offsets]


@pytest.mark.parametrize("n", range(1, 18))
def test_bruck_and_definition_agree(n):
    x = RNG.integers(-100, 100, size=(n, 3)).astype(np.int32)
    held, _ = bruck.allgather(list(x))
    ref = D.allgather(x)
    for r in range(n):
        assert sorted(held[r]) == list(range(n))
        for c in range(n):
            assert (held[r][c] == x[c]).all()
            assert (ref[r, c] == x[c]).all()


def reversed_bruck(n):
    """Dimension-reversed Bruck, built directly: at distance d (largest
    first) the positions that already hold the data are the multiples of 2d."""
    L = pat.ceil_log2(n)
    out = []
    d = 1 << (L - 1) if L else 0
    while d >= 1:
        out.append((d, [p for p in range(0, n, 2 * d) if p + d < n]))
        d //= 2
    return out


def test_farthest_first_n8_third_step_sends_four_chunks():
    g = read_golden("farthest_first_n8.txt")
    s = pat.schedule(8, full_t(8))
    assert [d for d, _ in s] == [int(v) for v in g["distances"]]
    assert [len(P) for _, P in s] == [int(v) for v in g["chunks_per_step"]]
    # the 4 chunks of the third step come from 4 different trees (ranks)
    r = 5
    assert len({(r - p) % 8 for p in s[2][1]}) == 4


def test_truncated_n7():
    g = read_golden("truncated_n7.txt")
    s = pat.schedule(7, full_t(7))
    assert [len(P) for _, P in s] == [int(v) for v in g["chunks_per_step"]]
    d2, P2 = s[1]
    assert d2 == 2 and sorted(-p for p in P2) == sorted(int(v) for v in g["step2_offsets"])
    d3, P3 = s[2]
    assert d3 == 1 and int(g["step3_includes_offset"][0]) in [-p for p in P3]
    # edges of rank 0's tree on the last step: position p is rank p
    edges = {f"{p}>{p + d3}" for p in P3}
    assert edges == set(g["tree0_last_step_edges"])


# --------------------------------------------------------------------------
# Section "The PAT algorithm": aggregation limit, linear part
# --------------------------------------------------------------------------

def test_pat_n8_aggregation_two():
    g = read_golden("pat_n8_agg2.txt")
    s = pat.schedule(8, 1)  # T = 2
    top = [st for st in s if st[0] >= 4]      # M = 8 / T = 4: distances >= 4 are the top
    lin = [st for st in s if st[0] < 4]
    assert len(top) == int(g["top_steps"][0])
    assert len(lin) == int(g["linear_steps"][0])
    assert max(len(P) for _, P in s) == int(g["max_chunks_per_step"][0])
    # the Bruck last step (distance 1, 4 chunks) is split in two, far part first
    last = [P for d, P in s if d == 1]
    assert len(last) == 2 and sorted(last[0] + last[1]) == [0, 2, 4, 6]
    assert min(last[0]) > min(last[1])
    # reading (far-first pre-order walk): the exact table
    assert s == [(4, [0]), (2, [0, 4]), (1, [2, 6]), (1, [0, 4])]


def test_pat_n16_transition():
    g = read_golden("pat_n16.txt")
    T_full = int(g["full_aggregation_trees"][0])
    assert pat.schedule(16, int(math.log2(T_full))) == reversed_bruck(16)
    counts = [len(pat.schedule(16, int(math.log2(int(T))))) for T in g["trees"]]
    # derived (the figures are missing): t top steps + (16 / T) - 1 linear steps
    assert counts == [4, 5, 8]


@pytest.mark.parametrize("n", [3, 5, 6, 7, 9, 12, 16, 23, 24, 31, 33, 64, 100])
def test_full_aggregation_is_reversed_bruck(n):
    assert pat.schedule(n, full_t(n)) == reversed_bruck(n)


def test_fully_linear_n8():
    g = read_golden("linear_n8.txt")
    assert int(g["trees"][0]) == 1
    s = pat.schedule(8, 0)
    assert len(s) == int(g["steps"][0])
    assert all(len(P) == 1 for _, P in s)


@pytest.mark.parametrize("n", range(2, 41))
def test_linear_steps_and_formula(n):
    L = pat.ceil_log2(n)
    assert len(pat.schedule(n, 0)) == n - 1  # one tree edge per step
    for t in range(L):
        s = pat.schedule(n, t)
        assert sum(len(P) for _, P in s) == n - 1  # every tree edge exactly once
        M = 1 << (L - t)
        assert len(s) == t + min(M, n) - 1


# --------------------------------------------------------------------------
# Abstract: exactly-once, logarithmic steps, logarithmic buffers
# --------------------------------------------------------------------------

@pytest.mark.parametrize("n", list(range(1, 34)) + [47, 64])
def test_exactly_once_every_aggregation(n):
    x = np.arange(n, dtype=np.int32).reshape(n, 1)  # chunk c carries its id
    for t in range(max(pat.ceil_log2(n), 1)):
        recv, _ = pat.allgather(x, t)  # the executor raises on a duplicate or a miss
        assert (recv[:, :, 0] == np.arange(n)[None, :]).all()


def test_log_steps_for_small_sizes():
    for n in list(range(2, 300)) + [999, 1000, 1001, 1024, 1025]:
        assert len(pat.schedule(n, full_t(n))) == pat.ceil_log2(n)
    assert len(pat.schedule(1000, full_t(1000))) == 10


@pytest.mark.parametrize("n", [2, 3, 5, 6, 7, 8, 11, 16, 24, 29, 32])
def test_log_buffers_independent_of_size(n):
    L = pat.ceil_log2(n)
    for t in range(max(L, 1)):
        T = 1 << t
        stats = []
        for m in (1, 17):
            x = RNG.integers(0, 9, size=(n, m)).astype(np.int32)
            _, st = pat.allgather(x, t)
            y = RNG.integers(0, 9, size=(n, n, m)).astype(np.int32)
            _, st2 = pat.reducescatter(y, t, "int32")
            stats.append((st["peak_per_dim"], st2["peak_per_dim"]))
            for peak in (st["peak_per_dim"], st2["peak_per_dim"]):
                assert len(peak) <= L  # at most one buffer per dimension
                assert all(v <= T for v in peak.values())  # each holds <= T chunks
        assert stats[0] == stats[1]  # same use at any size


def test_aggregation_level_fits_budget():
    for n in [6, 24, 64, 128, 1000, 37]:
        L = pat.ceil_log2(n)
        for chunk in [256, 4096, 65536, 1 << 20, 8 << 20]:
            for budget in [4096, 1 << 20, 8 << 20]:
                t = pat.aggregation_level(n, chunk, budget)
                k = max(len(P) for _, P in pat.schedule(n, t))
                if t > 0:
                    assert k * chunk <= budget
                if t < L - 1:
                    k2 = max(len(P) for _, P in pat.schedule(n, t + 1))
                    assert k2 * chunk > budget
    # the five workloads at an 8 MiB budget (float32 slots for bf16 reduce-scatter)
    mib = 1 << 20
    assert len(pat.schedule(6, pat.aggregation_level(6, 4096, 8 * mib))) == 3
    assert len(pat.schedule(24, pat.aggregation_level(24, 65536, 8 * mib))) == 5
    assert len(pat.schedule(64, pat.aggregation_level(64, mib, 8 * mib))) == 10
    assert len(pat.schedule(1000, pat.aggregation_level(1000, 256, 8 * mib))) == 10
    assert len(pat.schedule(128, pat.aggregation_level(128, 8 * mib, 8 * mib))) == 127


# --------------------------------------------------------------------------
# Brute force on tiny N; closed form of the reversed-tree association
# --------------------------------------------------------------------------

def closed_form(inputs, dtype):
    return pat.reducescatter_closed_form(inputs, dtype)


def _symbolic(n, root):
    """The closed form evaluated on names instead of numbers."""
    names = [f"x{(root + q) % n}" for q in range(n)]
    out = pat.reversed_tree_sum(names, n, lambda a, b: f"({a}+{b})")
    return out[1:-1] if out.startswith("(") and n > 1 else out


def test_closed_form_association_matches_hand_derivation():
    """The reversed-tree association written out by hand from the
    reduce-scatter section (tests/golden/rs_association.txt), for truncated
    and full trees and shifted roots."""
    g = read_golden("rs_association.txt")
    assert len(g) >= 9
    for key, (want,) in g.items():
        n, root = (int(v) for v in key[1:].split("_root"))
        assert _symbolic(n, root) == want, key


@pytest.mark.parametrize("n", [1, 2, 3, 6, 7, 13, 64, 100])
def test_closed_form_int32_is_the_plain_sum(n):
    """Integer adds associate: the closed form must equal the definition,
    which catches a dropped, doubled or misplaced term."""
    x = RNG.integers(-2**31, 2**31, size=(n, n, 5), dtype=np.int64).astype(np.int32)
    assert (closed_form(x, "int32") == D.reducescatter_sum(x, "int32")).all()
    f = np.zeros((n, n, 1), dtype=np.int64)
    for s in range(n):
        f[s] = 1 << (s % 31)
    if n <= 31:
        assert (closed_form(f.astype(np.int32), "int32").astype(np.int64) & 0xFFFFFFFF == (1 << n) - 1).all()


@pytest.mark.parametrize("n", [5, 24, 128, 1000])
def test_closed_form_error_bound(n):
    """|closed form - exact| <= gamma_L * sum|v| (Higham, section 4.2)."""
    x = RNG.standard_normal((n, n, 3)).astype(np.float32)
    got = closed_form(x, "float32").astype(np.float64)
    L = pat.ceil_log2(n)
    gamma = L * 2.0 ** -24 / (1 - L * 2.0 ** -24)
    assert (np.abs(got - D.reducescatter_sum(x, "float32")) <= gamma * D.reducescatter_abs_sum(x, "float32")).all()


def bf16_inputs(shape):
    return D.f32_to_bf16_bits(RNG.standard_normal(shape).astype(np.float32))


@pytest.mark.parametrize("n", range(1, 9))
@pytest.mark.parametrize("m", [1, 2, 3, 17])
def test_brute_force_small(n, m):
    for t in range(max(pat.ceil_log2(n), 1)):
        xa = RNG.integers(-2**31, 2**31, size=(n, m), dtype=np.int64).astype(np.int32)
        recv, _ = pat.allgather(xa, t)
        assert (recv == D.allgather(xa)).all()
        xb = bf16_inputs((n, m))
        recv, _ = pat.allgather(xb, t)
        assert (recv.view(np.uint16) == D.allgather(xb)).all()

        xi = RNG.integers(-2**31, 2**31, size=(n, n, m), dtype=np.int64).astype(np.int32)
        out, _ = pat.reducescatter(xi, t, "int32")
        assert (out == D.reducescatter_sum(xi, "int32")).all()

        xf = RNG.standard_normal((n, n, m)).astype(np.float32)
        out, _ = pat.reducescatter(xf, t, "float32")
        assert (out.view(np.uint32) == closed_form(xf, "float32").view(np.uint32)).all()

        xh = bf16_inputs((n, n, m))
        out, _ = pat.reducescatter(xh, t, "bfloat16")
        assert (out == closed_form(xh, "bfloat16")).all()


@pytest.mark.parametrize("n", [9, 13, 24, 31, 40])
def test_each_input_counted_once(n):
    """Formal sums: rank x contributes 2^x, so the sum names its terms."""
    m = 2
    x = np.zeros((n, n, m), dtype=np.int64)
    for s in range(n):
        x[s] = 1 << (s % 31)
    for t in range(pat.ceil_log2(n)):
        if n <= 31:
            out, _ = pat.reducescatter(x.astype(np.int32), t, "int32")
            assert (out.astype(np.int64) & 0xFFFFFFFF == (1 << n) - 1).all()
        y = RNG.integers(-2**20, 2**20, size=(n, n, m)).astype(np.int32)
        out, _ = pat.reducescatter(y, t, "int32")
        assert (out == D.reducescatter_sum(y, "int32")).all()


@pytest.mark.parametrize("n", [3, 6, 12, 24, 33])
def test_fp32_order_does_not_depend_on_aggregation(n):
    x = RNG.standard_normal((n, n, 64)).astype(np.float32)
    outs = [pat.reducescatter(x, t, "float32")[0] for t in range(pat.ceil_log2(n))]
    for o in outs[1:]:
        assert (o.view(np.uint32) == outs[0].view(np.uint32)).all()
    assert (outs[0].view(np.uint32) == closed_form(x, "float32").view(np.uint32)).all()


@pytest.mark.parametrize("n,dtype", [(6, "float32"), (24, "float32"), (64, "float32"),
                                     (24, "bfloat16"), (64, "bfloat16")])
def test_error_bound(n, dtype):
    """|tree sum - exact| <= gamma_L * sum|v| (each term passes through at most
    L = ceil(log2 N) float32 additions; Higham, Accuracy and Stability of
    Numerical Algorithms, section 4.2), plus one bf16 rounding of the result."""
    m = 257
    if dtype == "float32":
        x = RNG.standard_normal((n, n, m)).astype(np.float32)
    else:
        x = bf16_inputs((n, n, m))
    t = pat.aggregation_level(n, m * 4, 8 * 4 * m)
    out, _ = pat.reducescatter(x, t, dtype)
    exact = D.reducescatter_sum(x, dtype)
    scale = D.reducescatter_abs_sum(x, dtype)
    L = pat.ceil_log2(n)
    u = 2.0 ** -24
    gamma = L * u / (1 - L * u)
    if dtype == "float32":
        got = out.astype(np.float64)
        assert (np.abs(got - exact) <= gamma * scale).all()
    else:
        got = D.bf16_bits_to_f32(out).astype(np.float64)
        assert (np.abs(got - exact) <= gamma * scale + 2.0 ** -8 * np.abs(got)).all()
    assert (np.abs(got - exact) <= (1e-5 if dtype == "float32" else 1e-2) * scale).all()


def test_special_cases():
    # one rank: identity
    x = RNG.standard_normal((1, 1, 5)).astype(np.float32)
    out, st = pat.reducescatter(x, 0, "float32")
    assert st["steps"] == 0 and (out == x[0]).all()
    recv, st = pat.allgather(x[0], 0)
    assert st["steps"] == 0 and (recv == x[0][None]).all()
    # two ranks: one step, one add
    x = RNG.standard_normal((2, 2, 5)).astype(np.float32)
    out, st = pat.reducescatter(x, 0, "float32")
    assert st["steps"] == 1
    assert (out[0] == (x[0, 0] + x[1, 0]).astype(np.float32)).all()
    assert (out[1] == (x[1, 1] + x[0, 1]).astype(np.float32)).all()
    # empty chunks
    out, _ = pat.reducescatter(np.zeros((5, 5, 0), np.int32), 1, "int32")
    assert out.shape == (5, 0)
    recv, _ = pat.allgather(np.zeros((5, 0), np.float32), 1)
    assert recv.shape == (5, 5, 0)


def test_definitions_themselves():
    x = np.array([[[2**31 - 1], [1]], [[1], [-5]]], dtype=np.int32)
    out = D.reducescatter_sum(x, "int32")
    assert out[0, 0] == -2**31 and out[1, 0] == -4  # two's complement wrap
    b = D.f32_to_bf16_bits(np.array([1.0, 1.00390625, 1.01171875, -2.5], np.float32))
    assert list(b) == [0x3F80, 0x3F80, 0x3F82, 0xC020]  # ties to even
    assert list(D.bf16_bits_to_f32(b)) == [1.0, 1.0, 1.015625, -2.5]


# --------------------------------------------------------------------------
# Planted mistakes: each must make one of the pins above fail
# --------------------------------------------------------------------------

def breadth_first_walk(span):
    order, level = [], [0]
    d = span // 2
    while d >= 1:
        order += [(q, d) for q in level]
        level = level + [q + d for q in level]
        d //= 2
    return order


def test_planted_breadth_first_walk_breaks_buffer_bound(monkeypatch):
    monkeypatch.setattr(pat, "far_first_walk", breadth_first_walk)
    x = np.arange(8, dtype=np.int32).reshape(8, 1)
    _, st = pat.allgather(x, 0)
    assert max(st["peak_per_dim"].values()) > 1  # T = 1 bound violated


def test_planted_missing_truncation_is_caught(monkeypatch):
    def no_truncation(n, p, reach):
        return pat.ceil_log2(reach) if reach > 1 else 0
    monkeypatch.setattr(pat, "children", no_truncation)
    x = np.arange(7, dtype=np.int32).reshape(7, 1)
    with pytest.raises(AssertionError):
        pat.allgather(x, 2)


def test_planted_dropped_term_is_caught(monkeypatch):
    real = pat._add
    calls = {"n": 0}

    def drop_one(a, b, dtype):
        calls["n"] += 1
        return a if calls["n"] == 3 else real(a, b, dtype)
    monkeypatch.setattr(pat, "_add", drop_one)
    y = RNG.integers(1, 100, size=(6, 6, 4)).astype(np.int32)
    out, _ = pat.reducescatter(y, 2, "int32")
    assert not (out == D.reducescatter_sum(y, "int32")).all()


def test_planted_wrong_tree_index_is_caught(monkeypatch):
    # for a power-of-two N the mirrored labelling p -> -p is itself a valid
    # tree; truncation (N = 7) is what exposes it
    monkeypatch.setattr(pat, "tree_of", lambda r, p, n: (r + p) % n)
    x = np.arange(7, dtype=np.int32).reshape(7, 1)
    with pytest.raises(AssertionError):
        pat.allgather(x, 1)
    y = RNG.integers(-9, 9, size=(7, 7, 1)).astype(np.int32)
    with pytest.raises(AssertionError):
        pat.reducescatter(y, 1, "int32")


def test_planted_wrong_direction_is_caught(monkeypatch):
    monkeypatch.setattr(pat, "peer_of", lambda r, d, n: (r - d) % n)
    x = np.arange(6, dtype=np.int32).reshape(6, 1)
    with pytest.raises(AssertionError):
        pat.allgather(x, 2)


def test_planted_near_first_walk_is_caught(monkeypatch):
    def near_first(span):  # pre-order, nearest child first: a different association
        order = []

        def walk(q, w):
            d = 1
            while d < w:
                order.append((q, d))
                walk(q + d, d)
                d *= 2
        walk(0, span)
        return order
    monkeypatch.setattr(pat, "far_first_walk", near_first)
    with pytest.raises(AssertionError):
        test_pat_n8_aggregation_two()
    x = RNG.standard_normal((8, 8, 64)).astype(np.float32)
    out, _ = pat.reducescatter(x, 0, "float32")
    assert not (out.view(np.uint32) == closed_form(x, "float32").view(np.uint32)).all()


def test_planted_ring_order_association_is_caught(monkeypatch):
    def ring(values, n, add):  # rank after rank, as a ring would add them
        acc = values[0]
        for q in range(1, n):
            acc = add(acc, values[q])
        return acc
    monkeypatch.setattr(pat, "reversed_tree_sum", ring)
    with pytest.raises(AssertionError):
        test_closed_form_association_matches_hand_derivation()


def test_planted_far_child_first_association_is_caught(monkeypatch):
    def far_first(values, n, add):  # a node adds its farthest child first
        L = pat.ceil_log2(n)

        def S(lo, w):
            acc = values[lo]
            d = w // 2
            while d >= 1:
                if lo + d < n:
                    acc = add(acc, S(lo + d, d))
                d //= 2
            return acc
        return S(0, 1 << L)
    monkeypatch.setattr(pat, "reversed_tree_sum", far_first)
    with pytest.raises(AssertionError):
        test_closed_form_association_matches_hand_derivation()


def test_planted_mirrored_positions_in_closed_form_are_caught(monkeypatch):
    monkeypatch.setattr(pat, "rank_at", lambda root, q, n: (root - q) % n)
    x = RNG.standard_normal((7, 7, 64)).astype(np.float32)
    out, _ = pat.reducescatter(x, 1, "float32")
    assert not (out.view(np.uint32) == closed_form(x, "float32").view(np.uint32)).all()


# --------------------------------------------------------------------------
# The close-first linear order (section "The PAT algorithm": the alternative
# schedule that sends close first, then far)
# --------------------------------------------------------------------------

def test_close_first_n8_aggregation_two():
    # reading (close-first pre-order walk): same edges per step as far-first,
    # the linear part taken nearest child first
    s = pat.schedule(8, 1, "close")
    assert s == [(4, [0]), (1, [0, 4]), (2, [0, 4]), (1, [2, 6])]
    assert sorted(map(str, s)) == sorted(map(str, pat.schedule(8, 1, "far")))


@pytest.mark.parametrize("n", list(range(2, 34)) + [47, 64])
def test_close_first_invariants(n):
    L = pat.ceil_log2(n)
    for t in range(L):
        T = 1 << t
        far, close = pat.schedule(n, t, "far"), pat.schedule(n, t, "close")
        assert len(far) == len(close)  # same step count
        assert sorted(map(str, far)) == sorted(map(str, close))  # same steps, other order
        x = np.arange(n, dtype=np.int32).reshape(n, 1)
        recv, st = pat.allgather(x, t, "close")  # exactly once, checked inside
        assert (recv[:, :, 0] == np.arange(n)[None, :]).all()
        assert all(v <= T for v in st["peak_per_dim"].values())
        y = RNG.integers(-2**31, 2**31, size=(n, n, 3), dtype=np.int64).astype(np.int32)
        out, st2 = pat.reducescatter(y, t, "int32", "close")
        assert (out == D.reducescatter_sum(y, "int32")).all()
        assert all(v <= T for v in st2["peak_per_dim"].values())


@pytest.mark.parametrize("n", [6, 24, 33])
def test_close_first_fp32_error_bound(n):
    x = RNG.standard_normal((n, n, 129)).astype(np.float32)
    L = pat.ceil_log2(n)
    exact = D.reducescatter_sum(x, "float32")
    scale = D.reducescatter_abs_sum(x, "float32")
    gamma = L * 2.0 ** -24 / (1 - L * 2.0 ** -24)
    for t in range(L):
        out, _ = pat.reducescatter(x, t, "float32", "close")
        # each term still passes through at most L adds (the tree's depth)
        assert (np.abs(out.astype(np.float64) - exact) <= gamma * scale).all()
