"""The library's host schedule (C++) against the oracle's (Python), and a
symbolic execution of the library's step tables, slot indices included.

Integer work: every comparison is exact.  No GPU needed.
"""

import numpy as np
import pytest
from hypothesis import given, settings, strategies as hs

from oracle import pat as opat
from paper_2506_20252_amd import pat

NS = list(range(1, 70)) + [100, 127, 128, 129, 255, 256, 257, 1000]


def library_steps(coll, n, count, dtype):
    st, steps, entries = pat.pat_plan_steps(coll, n, count, dtype)
    assert st == pat.PAT_OK
    out, j = [], 0
    for d, k in steps:
        out.append((d, [e[0] for e in entries[j:j + k]]))
        j += k
    return out, steps, entries


def budget_for(n, t, chunk_bytes):
    """A budget that makes the library choose aggregation level t."""
    k = max(len(P) for _, P in opat.schedule(n, t))
    return k * chunk_bytes


@pytest.mark.parametrize("order", ["far", "close"])
@pytest.mark.parametrize("n", NS)
def test_schedule_matches_oracle_all_levels(n, order):
    L = opat.ceil_log2(n)
    count = 64  # float32: 256-byte chunks
    pat.check(pat.pat_set_linear_order(order))
    try:
        for t in range(max(L, 1)):
            pat.pat_set_buffer_bytes(budget_for(n, t, count * 4) if n > 1 else 1 << 20)
            ag, _, _ = library_steps(pat.PAT_ALLGATHER, n, count, "float32")
            rs, _, _ = library_steps(pat.PAT_REDUCESCATTER, n, count, "float32")
            want_t = opat.aggregation_level(n, count * 4, pat.pat_get_buffer_bytes())
            ref = opat.schedule(n, want_t, order)
            assert ag == [(d, sorted(P)) for d, P in ref]
            assert rs == [(d, sorted(P)) for d, P in reversed(ref)]
            if n > 2:
                assert want_t == t or len(opat.schedule(n, want_t)) == len(opat.schedule(n, t))
    finally:
        pat.pat_set_buffer_bytes(0)
        pat.pat_set_linear_order("far")


@pytest.mark.parametrize("n,count,dtype", [(6, 1024, "int32"), (24, 32768, "bfloat16"),
                                           (64, 262144, "float32"), (1000, 64, "float32"),
                                           (128, 2 << 20, "bfloat16"), (37, 5000, "float32")])
def test_aggregation_level_matches_oracle(n, count, dtype):
    for coll in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER):
        st, info = pat.pat_plan_info(coll, n, count, dtype)
        slot_bytes = count * (4 if (coll == pat.PAT_REDUCESCATTER or dtype != "bfloat16") else 2)
        t = opat.aggregation_level(n, slot_bytes, pat.pat_get_buffer_bytes())
        assert info["t"] == t
        assert info["steps"] == len(opat.schedule(n, t))


def children(n, pos, reach):
    c, d = 0, reach // 2
    while d >= 1:
        if pos + d < n:
            c += 1
        d //= 2
    return c


def run_symbolic_allgather(n, steps, entries):
    """Execute the library's all-gather table on symbols: slots hold
    (chunk, forwards left), receive buffers record arrivals."""
    slots = {}
    got = [{r} for r in range(n)]
    peak = 0
    j = 0
    for d, k in steps:
        writes = []
        for r in range(n):
            for (p, a, b, _c) in entries[j:j + k]:
                c = (r - p) % n
                if a == -1:
                    assert p == 0
                else:
                    held = slots.get((r, a))
                    assert held is not None and held[0] == c and held[1] > 0, "read of a slot not holding the chunk"
                    held[1] -= 1
                peer = (r + d) % n
                writes.append((peer, c, b, children(n, p + d, d)))
        for peer, c, b, fwd in writes:
            assert c not in got[peer], "chunk received twice"
            got[peer].add(c)
            if b >= 0:
                old = slots.get((peer, b))
                assert old is None or old[1] == 0, "slot overwritten before it was drained"
                assert fwd > 0
                slots[(peer, b)] = [c, fwd]
            else:
                assert fwd == 0, "a forwarding receiver got no slot"
        live = {}
        for (rank, _), v in slots.items():
            if v[1] > 0:
                live[rank] = live.get(rank, 0) + 1
        peak = max([peak] + list(live.values()))
        j += k
    assert all(got[r] == set(range(n)) for r in range(n))
    assert all(v[1] == 0 for v in slots.values())
    return peak


def run_symbolic_reducescatter(n, steps, entries):
    """Execute the library's reduce-scatter table on formal sums (sets of
    contributing ranks), checking every slot read and write."""
    slots = {}   # (rank, slot) -> [tree, position, set of ranks]
    root = {}    # rank -> set of ranks
    last_root = max(j for j, e in enumerate(entries) if e[0] == 0)
    seen = set()  # positions that have received already (the same for every rank)
    j = 0
    for d, k in steps:
        ops = []
        first = {}
        for jj, (p, _a, _b, _c) in enumerate(entries[j:j + k]):
            first[jj] = p not in seen
            seen.add(p)
        for r in range(n):
            for jj, (p, a, b, c) in enumerate(entries[j:j + k]):
                tree = (r - p) % n
                child = (r + d) % n
                if a == -1:
                    assert children(n, p + d, d) == 0, "a non-leaf child sent its raw input"
                    part = {child}
                else:
                    held = slots.get((child, a))
                    assert held is not None and held[0] == tree and held[1] == p + d
                    part = held[2]
                    slots[(child, a)] = None  # drained
                ops.append((r, p, tree, b, c, part, first[jj], j + jj == last_root))
        for r, p, tree, b, c, part, is_first, is_last_root in ops:
            assert (b == -1) == is_first, "own input must enter exactly at the first receive"
            if b == -1:
                own = {r}
            elif b == -2:
                assert p == 0 and r in root
                own = root[r]
            else:
                held = slots.get((r, b))
                assert held is not None and held[0] == tree and held[1] == p
                own = held[2]
            assert not (own & part), "a contribution counted twice"
            total = own | part
            if c in (-2, -3):
                assert p == 0 and tree == r
                assert (c == -3) == is_last_root
                root[r] = total
            else:
                old = slots.get((r, c))
                assert old is None or (old[0] == tree and old[1] == p), "live slot overwritten"
                slots[(r, c)] = [tree, p, total]
        j += k
    assert all(root[r] == set(range(n)) for r in range(n))
    assert all(v is None for v in slots.values())


@pytest.mark.parametrize("order", ["far", "close"])
@pytest.mark.parametrize("n", list(range(2, 34)) + [47, 64, 100])
def test_symbolic_execution_of_library_tables(n, order):
    L = opat.ceil_log2(n)
    pat.check(pat.pat_set_linear_order(order))
    try:
        for t in range(L):
            pat.pat_set_buffer_bytes(budget_for(n, t, 256))
            _, steps, entries = library_steps(pat.PAT_ALLGATHER, n, 64, "float32")
            peak = run_symbolic_allgather(n, steps, entries)
            T = 1 << t
            assert peak <= L * T
            _, steps, entries = library_steps(pat.PAT_REDUCESCATTER, n, 64, "float32")
            run_symbolic_reducescatter(n, steps, entries)
            st, info = pat.pat_plan_info(pat.PAT_ALLGATHER, n, 64, "float32")
            assert info["slot_dims"] <= L and info["slot_chunks_per_rank"] <= L * T
    finally:
        pat.pat_set_buffer_bytes(0)
        pat.pat_set_linear_order("far")


def _slot_trees(coll, n, steps, entries, lo, hi):
    """(rank, slot entry) -> set of trees that launch-level steps [lo, hi) touch there."""
    use = {}
    j = 0
    for s, (d, k) in enumerate(steps):
        if lo <= s < hi:
            for (p, a, b, c) in entries[j:j + k]:
                for r in range(n):
                    tree = (r - p) % n
                    if coll == pat.PAT_REDUCESCATTER:
                        touched = [((r + d) % n, a), (r, b), (r, c)]
                    else:
                        touched = [(r, a), ((r + d) % n, b)]
                    for rank, slot in touched:
                        if slot >= 0:
                            use.setdefault((rank, slot), set()).add(tree)
        j += k
    return use


@pytest.mark.parametrize("order", ["far", "close"])
@pytest.mark.parametrize("n", [3, 4, 5, 7, 8, 9, 16, 24, 33, 64, 100, 129])
def test_top_part_slots_serve_one_tree(n, order):
    """What fusing the top part relies on: in the top t steps (the first t of
    the all-gather, the last t of the reduce-scatter) every intermediate-buffer
    entry of every rank holds chunks of one tree only, so a workgroup that owns
    a tree may run those steps without waiting for other trees.  The linear
    part, by contrast, reuses entries across trees once T < 2^(L-1)."""
    count = 64
    pat.check(pat.pat_set_linear_order(order))
    try:
        saw_linear_reuse = False
        L = opat.ceil_log2(n)
        for t in range(1, max(L, 1)):
            pat.pat_set_buffer_bytes(budget_for(n, t, count * 4))
            for coll in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER):
                st, info = pat.pat_plan_info(coll, n, count, "float32")
                assert st == pat.PAT_OK and info["pieces"] == 1
                _, steps, entries = library_steps(coll, n, count, "float32")
                ns, tt = len(steps), info["t"]
                lo, hi = (0, tt) if coll == pat.PAT_ALLGATHER else (ns - tt, ns)
                assert all(d >= 1 << (L - tt) for d, _ in steps[lo:hi])  # the fully aggregated distances
                top = _slot_trees(coll, n, steps, entries, lo, hi)
                assert all(len(trees) == 1 for trees in top.values()), (coll, t)
                rest = (hi, ns) if coll == pat.PAT_ALLGATHER else (0, lo)
                lin = _slot_trees(coll, n, steps, entries, *rest)
                saw_linear_reuse |= any(len(trees) > 1 for trees in lin.values())
        if L >= 4:  # t = 1 leaves sub-trees of span >= 8, whose distance-2 entries serve two trees
            assert saw_linear_reuse
    finally:
        pat.pat_set_buffer_bytes(0)
        pat.pat_set_linear_order("far")


def test_top_fusion_setting_roundtrip():
    assert pat.pat_get_top_fusion() == pat.PAT_FUSION_AUTO
    for m in ("on", "off", "auto"):
        assert pat.pat_set_top_fusion(m) == pat.PAT_OK
        assert pat.pat_get_top_fusion() == pat.FUSIONS[m]
    assert pat.pat_set_top_fusion(7) == pat.PAT_ERR_INVALID_ARGUMENT
    assert pat.pat_get_top_fusion() == pat.PAT_FUSION_AUTO


@pytest.mark.parametrize("coll", [pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER])
def test_fused_range_reported_by_plan_info(coll):
    """Which steps run as one fused launch (stream and graph modes).  Both
    plans are fully aggregated, so every step may fuse: N=1000 with 256-byte
    chunks fuses (AUTO) the 8 narrow far steps, with at most 125 chunks per
    rank (the next moves 3 x 1000 x 250 x 256 B, over the 128 MiB limit),
    or (ON) all 10; N=6 with 4 KiB chunks all 3 steps.  A plan
    with a wider linear part fuses its top part only, and a top part of one
    step is never fused."""
    try:
        for fusion, want in (("auto", (8, 3)), ("on", (10, 1)), ("off", (0, 10))):
            pat.check(pat.pat_set_top_fusion(fusion))
            st, info = pat.pat_plan_info(coll, 1000, 64, "float32")
            assert st == pat.PAT_OK and info["steps"] == 10 and info["t"] == 9
            assert (info["fused_steps"], info["launches_per_op"]) == want
        pat.check(pat.pat_set_top_fusion("auto"))
        st, info = pat.pat_plan_info(coll, 6, 1024, "int32")
        assert (info["t"], info["fused_steps"], info["launches_per_op"]) == (2, 3, 1)
        # N=64, 1 MiB float32 chunks: T = 8 sub-trees of span 8; ON fuses the 3 top steps
        pat.check(pat.pat_set_top_fusion("on"))
        st, info = pat.pat_plan_info(coll, 64, 1 << 18, "float32")
        assert (info["t"], info["steps"], info["fused_steps"], info["launches_per_op"]) == (3, 10, 3, 8)
        pat.check(pat.pat_set_top_fusion("auto"))
        # 4 MiB bf16 chunks: the all-gather's slots hold bf16 (T = 2, 64 steps, one top step),
        # the reduce-scatter's hold float32 partials (T = 1, 127 steps, no top part)
        st, info = pat.pat_plan_info(coll, 128, 2 << 20, "bfloat16")
        want = (1, 0, 64) if coll == pat.PAT_ALLGATHER else (0, 0, 127)
        assert (info["t"], info["fused_steps"], info["launches_per_op"]) == want
    finally:
        pat.check(pat.pat_set_top_fusion("auto"))


def test_streaming_choice_reported_by_plan_info(monkeypatch):
    """Operations of >= 1e9 algorithmic bytes stream (nontemporal accesses);
    smaller ones keep their slots cached between steps; PAT_STREAMING forces
    either."""
    for args, want in (((pat.PAT_REDUCESCATTER, 128, 2 << 20, "bfloat16"), 1),
                       ((pat.PAT_REDUCESCATTER, 64, 262144, "float32"), 1),
                       ((pat.PAT_REDUCESCATTER, 1000, 64, "float32"), 0),
                       ((pat.PAT_ALLGATHER, 24, 32768, "bfloat16"), 0)):
        st, info = pat.pat_plan_info(*args)
        assert st == pat.PAT_OK
        assert info["streaming"] == want, args
        assert (info["alg_bytes"] >= 1e9) == bool(want)
    # work order: a contiguous eighth per XCD for all-gathers (0), runs of 32 for reduce-scatters
    for args, want in (((pat.PAT_REDUCESCATTER, 128, 2 << 20, "bfloat16"), 32),
                       ((pat.PAT_REDUCESCATTER, 1000, 64, "float32"), 32),
                       ((pat.PAT_ALLGATHER, 64, 262144, "float32"), 0),
                       ((pat.PAT_ALLGATHER, 24, 32768, "bfloat16"), 0)):
        assert pat.pat_plan_info(*args)[1]["xcd_run"] == want, args
    monkeypatch.setenv("PAT_STREAMING", "1")
    assert pat.pat_plan_info(pat.PAT_ALLGATHER, 24, 32768, "bfloat16")[1]["streaming"] == 1
    monkeypatch.setenv("PAT_STREAMING", "0")
    assert pat.pat_plan_info(pat.PAT_REDUCESCATTER, 64, 262144, "float32")[1]["streaming"] == 0


@pytest.mark.parametrize("n", [2048, 4096, 4097])
def test_large_rank_counts_match_oracle(n):
    """Large N at full aggregation and at T = 1 (the two ends of the budget
    range): the library's steps equal the oracle's, ceil(log2 N) and N - 1."""
    count = 4
    L = opat.ceil_log2(n)
    try:
        for t in (L - 1, 0):
            pat.pat_set_buffer_bytes(budget_for(n, t, count * 4))
            for coll, rev in ((pat.PAT_ALLGATHER, False), (pat.PAT_REDUCESCATTER, True)):
                got, steps, _ = library_steps(coll, n, count, "float32")
                ref = [(d, sorted(P)) for d, P in opat.schedule(n, t)]
                assert got == (ref[::-1] if rev else ref)
                assert len(steps) == (L if t == L - 1 else n - 1)
    finally:
        pat.pat_set_buffer_bytes(0)


@pytest.mark.parametrize("order", ["far", "close"])
@pytest.mark.parametrize("n", [2, 3, 4, 5, 6, 7, 8, 9, 12, 16, 24, 33, 64, 100, 129, 1000])
def test_whole_schedule_slots_serve_one_tree_up_to_span_4(n, order):
    """When the sub-trees span M <= 4 every slot entry of the whole schedule
    serves one tree, linear part included: its distance-2 entry at index p / 4
    is used by position 4 idx + 2 alone, and leaves use no entry.  All steps
    may then run as one fused launch.  From span 8 on, the distance-2 entries
    of positions 8 idx + 2 and 8 idx + 6 are shared by two trees (unless
    truncation leaves 8 idx + 6 a leaf, as at N = 6 and 7)."""
    count = 64
    pat.check(pat.pat_set_linear_order(order))
    try:
        L = opat.ceil_log2(n)
        for t in range(max(L - 4, 0), max(L, 1)):
            pat.pat_set_buffer_bytes(budget_for(n, t, count * 4))
            for coll in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER):
                st, info = pat.pat_plan_info(coll, n, count, "float32")
                if info["t"] != t:
                    continue  # truncation made this budget reach the next level
                M = 1 << (L - t)
                _, steps, entries = library_steps(coll, n, count, "float32")
                use = _slot_trees(coll, n, steps, entries, 0, len(steps))
                one = all(len(trees) == 1 for trees in use.values())
                assert one == (M <= 4 or n in (6, 7)), (coll, t, M)
                if M <= 4 and len(steps) >= 2:
                    pat.check(pat.pat_set_top_fusion("on"))
                    _, fused = pat.pat_plan_info(coll, n, count, "float32")
                    pat.check(pat.pat_set_top_fusion("auto"))
                    assert fused["fused_steps"] == len(steps) and fused["launches_per_op"] == 1
    finally:
        pat.pat_set_buffer_bytes(0)
        pat.pat_set_linear_order("far")
        pat.check(pat.pat_set_top_fusion("auto"))


@settings(max_examples=60, deadline=None, derandomize=True)
@given(n=hs.integers(min_value=2, max_value=6000), level=hs.floats(min_value=0.0, max_value=1.0),
       order=hs.sampled_from(["far", "close"]))
def test_random_rank_counts_match_oracle(n, level, order):
    """Rank counts drawn over 2 .. 6000 (a fixed, derandomized draw), at an
    aggregation level drawn over 0 .. L-1: the library's steps equal the
    oracle's; there are t + M - 1 of them (sub-trees of span M = 2^(L-t),
    fewer when truncation empties a step), and they move N - 1 chunks per
    rank in all."""
    L = opat.ceil_log2(n)
    t = min(L - 1, int(level * L))
    count = 4
    pat.check(pat.pat_set_linear_order(order))
    try:
        pat.pat_set_buffer_bytes(budget_for(n, t, count * 4))
        st, info = pat.pat_plan_info(pat.PAT_ALLGATHER, n, count, "float32")
        assert st == pat.PAT_OK
        t = info["t"]  # truncation may let this budget reach the next level
        ref = [(d, sorted(P)) for d, P in opat.schedule(n, t, order)]
        got, steps, _ = library_steps(pat.PAT_ALLGATHER, n, count, "float32")
        assert got == ref
        got_rs, _, _ = library_steps(pat.PAT_REDUCESCATTER, n, count, "float32")
        assert got_rs == ref[::-1]
        assert sum(k for _, k in steps) == n - 1
        assert len(steps) <= t + (1 << (L - t)) - 1
        if n == 1 << L:
            assert len(steps) == t + (1 << (L - t)) - 1
    finally:
        pat.pat_set_buffer_bytes(0)
        pat.pat_set_linear_order("far")



@pytest.mark.parametrize("n,count,dtype,coll", [(65536, 1, "float32", pat.PAT_REDUCESCATTER),
                                                (65536, 1, "int32", pat.PAT_ALLGATHER),
                                                (1000, 64, "float32", pat.PAT_REDUCESCATTER),
                                                (24, 17, "bfloat16", pat.PAT_REDUCESCATTER),
                                                (128, 2 << 20, "bfloat16", pat.PAT_REDUCESCATTER)])
def test_slot_memory_follows_the_data(n, count, dtype, coll):
    """Intermediate memory per rank is the slot entries times the entry's own
    size when an entry is under 256 bytes (packed), else times its size
    rounded up to 256 bytes; bf16 reduce-scatters add one float32 root
    accumulator per rank.  At N = 65536 with one-element chunks that is 128 KiB
    per rank, not 32767 entries padded to 256 bytes (512 GiB in all)."""
    st, info = pat.pat_plan_info(coll, n, count, dtype)
    assert st == pat.PAT_OK
    entry = info["piece_elems"] * info["slot_elem_bytes"]
    stride = entry if entry < 256 else -(-entry // 256) * 256
    assert info["slot_bytes_per_rank"] == info["slot_chunks_per_rank"] * stride
    root = 0
    if coll == pat.PAT_REDUCESCATTER and dtype == "bfloat16":
        root_entry = info["piece_elems"] * 4
        root = root_entry if root_entry < 256 else -(-root_entry // 256) * 256
    assert info["slot_bytes_total"] == (info["slot_bytes_per_rank"] + root) * n
    if n == 65536:
        assert info["slot_bytes_per_rank"] == 32767 * 4


@pytest.mark.parametrize("coll", [pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER])
@pytest.mark.parametrize("dtype", ["int32", "float32", "bfloat16"])
def test_vector_path_reported_by_plan_info(coll, dtype):
    """The kernels a plan takes with 16-byte-aligned buffers, as the header
    states them: aligned vectors when every piece is whole vectors (16 bytes;
    bf16 reduce-scatter: 4 elements); else relaxed vectors when every piece
    holds at least one; else single elements.  Pieces come from small
    budgets, so the last piece may be under one vector while the others are
    not."""
    es = 2 if dtype == "bfloat16" else 4
    per = 4 if coll == pat.PAT_REDUCESCATTER else 16 // es  # elements per vector
    try:
        for budget in (0, 48, 100, 1000):
            pat.check(pat.pat_set_buffer_bytes(budget))
            for count in (1, 3, 4, 5, 7, 8, 9, 15, 16, 17, 63, 64, 65, 1000, 1001, 1003, 1004):
                st, info = pat.pat_plan_info(coll, 5, count, dtype)
                pat.check(st)
                pe, k = info["piece_elems"], info["pieces"]
                lens = [pe] * (k - 1) + [count - (k - 1) * pe]
                assert all(x > 0 for x in lens)
                whole = all(x % per == 0 for x in lens)
                holds_one = all(x >= per for x in lens)
                want = 1 if whole else 2 if holds_one else 0
                assert info["vector_path"] == want, (budget, count, lens)
    finally:
        pat.check(pat.pat_set_buffer_bytes(0))


@pytest.mark.parametrize("n", [5, 6, 7, 12, 13, 16, 24, 33, 64, 100, 128])
@pytest.mark.parametrize("K", [3, 5, 6, 7])
def test_list_schedule_of_budget_aggregation(n, K):
    """PAT_AGGREGATION_BUDGET with a budget of K chunks per step (K not a
    power of two): where the library takes its list schedule, the tables
    never need more steps than the power-of-two schedule, never carry more
    than K chunks per step or hold more than K per slot, pass the symbolic
    execution, and -- run by the oracle's own step executors, which check
    every transfer -- deliver every chunk exactly once and sum in the same
    association as the reversed-tree closed form."""
    count, esize = 17, 4
    rng = np.random.default_rng(n * 10 + K)
    pat.check(pat.pat_set_buffer_bytes(K * count * esize))
    try:
        pat.check(pat.pat_set_aggregation("pow2"))
        pow2 = {c: pat.pat_plan_info(c, n, count, "float32")[1]["steps"]
                for c in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER)}
        pat.check(pat.pat_set_aggregation("budget"))
        for coll in (pat.PAT_ALLGATHER, pat.PAT_REDUCESCATTER):
            st, info = pat.pat_plan_info(coll, n, count, "float32")
            st, steps, entries = pat.pat_plan_steps(coll, n, count, "float32")
            assert len(steps) == info["steps"] <= pow2[coll]
            assert max(k for _, k in steps) <= K
            if coll == pat.PAT_ALLGATHER:
                run_symbolic_allgather(n, steps, entries)  # its peak sums every slot of a rank
                ag_steps, j = [], 0
                for d, k in steps:
                    ag_steps.append((d, sorted(e[0] for e in entries[j:j + k])))
                    j += k
                x = rng.integers(-2**31, 2**31, size=(n, 3), dtype=np.int64).astype(np.int32)
                recv, stats = opat.allgather(x, 0, steps=ag_steps)
                assert (recv == np.broadcast_to(x[None], (n,) + x.shape)).all()
                assert max(stats["peak_per_dim"].values(), default=0) <= K
                xf = rng.standard_normal((n, n, 5)).astype(np.float32)
                out, stats = opat.reducescatter(xf, 0, "float32", steps=ag_steps)
                assert (out.view(np.uint32) == opat.reducescatter_closed_form(xf, "float32").view(np.uint32)).all()
                assert max(stats["peak_per_dim"].values(), default=0) <= K
                list_ag = info["list_schedule"]
            else:
                run_symbolic_reducescatter(n, steps, entries)
                assert info["list_schedule"] == list_ag
                assert info["fused_steps"] == 0 or not info["list_schedule"]
    finally:
        pat.check(pat.pat_set_aggregation("pow2"))
        pat.check(pat.pat_set_buffer_bytes(0))


def test_list_schedule_shortens_non_power_of_two_budgets():
    """The point of the list schedule: with 3 chunks per step, N = 128 needs
    fewer than the 64 steps of T = 2; with a power-of-two budget and a
    power-of-two N nothing changes."""
    pat.check(pat.pat_set_aggregation("budget"))
    try:
        pat.check(pat.pat_set_buffer_bytes(3 * 256))
        st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, 128, 64, "float32")
        assert info["list_schedule"] == 1 and info["steps"] < 64 and info["max_chunks_per_step"] <= 3
        pat.check(pat.pat_set_buffer_bytes(4 * 256))
        st, info = pat.pat_plan_info(pat.PAT_REDUCESCATTER, 128, 64, "float32")
        assert info["list_schedule"] == 0 and info["steps"] == 33
    finally:
        pat.check(pat.pat_set_aggregation("pow2"))
        pat.check(pat.pat_set_buffer_bytes(0))
