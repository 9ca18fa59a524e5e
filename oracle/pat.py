"""PAT (Parallel Aggregated Trees): schedule and step-by-step executors.

Test infrastructure only (see the package docstring).  Plain Python and numpy,
written from the paper's prose; every step names the passage it follows.

Model (section "Binomial-tree based algorithms"): the data of every rank x is
broadcast along its own binomial tree, shifted so that tree position q is rank
(x + q) mod N.  Data travels from rank r to rank r + d, d a power of two (the
"dimension" is log2 d).  With the farthest dimension first, the node reached
over distance D forwards over every smaller distance, farthest first; the root
behaves as if reached over 2^L, L = ceil(log2 N).  For a rank count that is
not a power of two the tree is truncated: an edge whose destination position
is N or more does not exist.

Steps (section "The PAT algorithm"): the intermediate buffer bounds how many
chunks a rank may send at once.  With T = 2^t parallel sub-trees the top t
dimensions are fully aggregated (one step per dimension, as in the
reversed-dimension Bruck algorithm); below that, the T sub-trees of span
M = 2^(L-t) each walk their edges one at a time, starting far and getting
closer, so that a buffer is emptied before its dimension is used again.  All T
sub-trees (and all N shifted trees) take the same walk step in parallel.

Reduce-scatter (section "Conversion to reduce-scatter operations") runs the
same steps in reverse order over reversed edges: close dimensions first,
parallel sub-trees first and the logarithmic top part last; each received
partial is added to the receiver's accumulation buffer, or, for the rank whose
own chunk it is, to its receive buffer.

Readings of points the paper leaves open (each one is listed with its reason in
the design notes; section numbers refer to the paper):

* direction: all-gather data moves r -> r + d, so rank r is position p of tree
  (r - p) mod N; reduce-scatter mirrors it (r + d -> r);
* the far-first linear walk is a pre-order walk of the sub-tree that takes the
  farthest child first (the breadth-first order breaks the buffer property);
* T is the largest power of two <= 2^(L-1) for which the largest step fits the
  buffer: (chunks of the largest step) * (chunk bytes) <= budget; a chunk
  larger than the budget runs with T = 1 (it is split into pieces, which does
  not change any result since both operations are elementwise);
* reduce-scatter: a leaf sends its raw input; a rank's own input enters at its
  first receive; the root accumulates in the receive buffer (a float32 copy of
  it for bfloat16 data, rounded once at the end).
"""

import numpy as np

from .definitions import bf16_bits_to_f32, f32_to_bf16_bits


def ceil_log2(n: int) -> int:
    L = 0
    while (1 << L) < n:
        L += 1
    return L


def lowbit(p: int) -> int:
    return p & -p


def tree_of(r: int, p: int, nranks: int) -> int:
    """The tree (= the rank whose chunk it carries) in which rank r sits at
    position p: positions count forward from the root, so it is r - p."""
    return (r - p) % nranks


def peer_of(r: int, d: int, nranks: int) -> int:
    """All-gather data travels forward: rank r sends over distance d to r + d."""
    return (r + d) % nranks


def rank_at(root: int, q: int, nranks: int) -> int:
    """The rank at position q of the tree rooted at `root` (the inverse of
    tree_of): positions count forward from the root."""
    return (root + q) % nranks


# --------------------------------------------------------------------------
# Trees and steps
# --------------------------------------------------------------------------

def tree_edges(nranks: int):
    """Edges (p, p + d, d) of one truncated binomial tree, farthest first.

    The root (position 0) holds the data.  A node reached over distance D
    forwards to p + d for d = D/2, D/4, ..., 1 when p + d < N (section
    "Binomial-tree based algorithms": farthest dimension first, truncated tree
    for non-power-of-two counts).  The list is in depth-first order, which is
    irrelevant here: steps are assigned per edge below.
    """
    L = ceil_log2(nranks)
    edges = []

    def grow(p, reach):
        d = reach // 2
        while d >= 1:
            if p + d < nranks:
                edges.append((p, p + d, d))
                grow(p + d, d)
            d //= 2

    if nranks > 1:
        grow(0, 1 << L)
    return edges


def far_first_walk(span: int):
    """Edges (q, d) of a full sub-tree of the given span, in the order the
    linear part sends them: from each node the farthest child first, and that
    child's whole sub-tree before the next, closer child (section "The PAT
    algorithm": start far, get closer, and empty each buffer before its
    dimension is used again)."""
    order = []

    def walk(q, w):
        d = w // 2
        while d >= 1:
            order.append((q, d))
            walk(q + d, d)
            d //= 2

    walk(0, span)
    return order


def close_first_walk(span: int):
    """The other linear order the paper allows (section "The PAT algorithm"):
    from each node the nearest child first, then farther ones, each child's
    whole sub-tree right after the edge that reached it (so each buffer is
    still drained before its dimension is used again)."""
    order = []

    def walk(q, w):
        d = 1
        while d < w:
            order.append((q, d))
            walk(q + d, d)
            d *= 2

    walk(0, span)
    return order


def schedule(nranks: int, t: int, order: str = "far"):
    """All-gather steps for N ranks and T = 2^t parallel sub-trees.

    Returns a list of (d, P): at that step every rank r sends, for each tree
    position p in P, chunk (r - p) mod N to rank (r + d) mod N.  Each edge of
    the relative tree is given a step: the top t dimensions (d >= M) get one
    fully aggregated step each, farthest first; an edge below the top belongs
    to sub-tree p // M and is sent at the position its relative edge
    (p mod M, d) has in the linear walk of a span-M sub-tree: far-first
    (order="far", the default) or close-first (order="close").  Positions that
    a truncated tree lacks simply send nothing; a step left with no edge does
    not exist.
    """
    if order not in ("far", "close"):
        raise ValueError(order)
    if nranks <= 1:
        return []
    L = ceil_log2(nranks)
    t = max(0, min(t, L - 1))
    M = 1 << (L - t)
    walk = far_first_walk(M) if order == "far" else close_first_walk(M)
    walk_index = {edge: i for i, edge in enumerate(walk)}
    groups = {}
    for p, _child, d in tree_edges(nranks):
        if d >= M:
            key = (0, L - 1 - (d.bit_length() - 1))
        else:
            key = (1, walk_index[(p % M, d)])
        groups.setdefault(key, (d, []))[1].append(p)
    return [(d, sorted(P)) for _, (d, P) in sorted(groups.items())]


def aggregation_level(nranks: int, chunk_bytes: int, budget_bytes: int) -> int:
    """t such that T = 2^t is the most sub-trees the budget permits (section
    "The PAT algorithm": aggregation limited to what the buffer holds)."""
    if nranks <= 1:
        return 0
    L = ceil_log2(nranks)
    best = 0
    for t in range(L):
        largest = max(len(P) for _, P in schedule(nranks, t))
        if largest * chunk_bytes <= budget_bytes:
            best = t
    return best


# --------------------------------------------------------------------------
# All-gather executor
# --------------------------------------------------------------------------

def children(nranks: int, p: int, reach: int) -> int:
    """How many times the node at position p, reached over `reach`, forwards."""
    n, d = 0, reach // 2
    while d >= 1:
        if p + d < nranks:
            n += 1
        d //= 2
    return n


def allgather(inputs: np.ndarray, t: int, order: str = "far", steps=None):
    """Execute the all-gather steps on per-rank data.

    inputs: (N, m) -- rank x's send buffer.  Returns (recv, stats): recv is
    (N, N, m) with recv[r][c] the chunk of rank c as received by rank r.

    A rank sends its own chunk from its send buffer; every other chunk it
    forwards comes from its intermediate buffer for the dimension it arrived
    on, where the transfer put it, and leaves that buffer after the last
    forward.  A chunk that will not be forwarded goes only to the receive
    buffer.  Every transfer is checked: the sender holds the chunk, the
    receiver never gets a chunk twice.

    `steps`, if given, replaces schedule(N, t, order): any list of (d, P) in
    the same form (e.g. another schedule under test), executed and checked the
    same way.
    """
    inputs = np.asarray(inputs)
    N = inputs.shape[0]
    recv = np.zeros((N,) + inputs.shape, dtype=inputs.dtype)
    have = np.zeros((N, N), dtype=bool)
    for r in range(N):  # own chunk: a local copy
        recv[r, r] = inputs[r]
        have[r, r] = True
    buf = [dict() for _ in range(N)]  # rank -> {(d, chunk): [data, forwards left]}
    peak = {}  # d -> most chunks any rank held for dimension d at once
    steps = schedule(N, t, order) if steps is None else steps
    for d, P in steps:
        messages = []
        for r in range(N):
            for p in P:
                c = tree_of(r, p, N)
                if p == 0:
                    data = inputs[r]
                else:
                    key = (lowbit(p), c)
                    if key not in buf[r]:
                        raise AssertionError(f"rank {r} forwards chunk {c} it does not hold")
                    entry = buf[r][key]
                    data = entry[0]
                    entry[1] -= 1
                    if entry[1] == 0:
                        del buf[r][key]
                messages.append((peer_of(r, d, N), c, p + d, data))
        for dst, c, pos, data in messages:
            if have[dst, c]:
                raise AssertionError(f"rank {dst} receives chunk {c} twice")
            recv[dst, c] = data
            have[dst, c] = True
            fwd = children(N, pos, d)
            if fwd:
                key = (d, c)
                if key in buf[dst]:
                    raise AssertionError("intermediate buffer entry overwritten")
                buf[dst][key] = [data, fwd]
        for r in range(N):
            held = {}
            for dd, _ in buf[r]:
                held[dd] = held.get(dd, 0) + 1
            for dd, n in held.items():
                peak[dd] = max(peak.get(dd, 0), n)
    if not have.all():
        raise AssertionError("some rank is missing a chunk")
    if any(buf[r] for r in range(N)):
        raise AssertionError("intermediate buffers not drained")
    stats = {"steps": len(steps), "chunks_per_step": [len(P) for _, P in steps],
             "peak_per_dim": peak}
    return recv, stats


# --------------------------------------------------------------------------
# Reduce-scatter executor
# --------------------------------------------------------------------------

def _widen(x, dtype):
    if dtype == "int32":
        return x.view(np.uint32).copy()  # wraparound adds
    if dtype == "float32":
        return x.astype(np.float32)
    if dtype == "bfloat16":
        return bf16_bits_to_f32(x)
    raise ValueError(dtype)


def _add(a, b, dtype):
    if dtype == "int32":
        return (a + b).astype(np.uint32)
    return (a + b).astype(np.float32)  # float32 + float32, one rounding


def reducescatter(inputs: np.ndarray, t: int, dtype: str, order: str = "far", steps=None):
    """Execute the reduce-scatter steps (reversed trees) on per-rank data.

    inputs: (N, N, m) -- inputs[x][c] is rank x's contribution to chunk c.
    Returns (out, stats): out is (N, m) in the input dtype.

    The all-gather steps are taken in reverse order and every edge reversed:
    at step (d, P) the rank r at position p of tree c = (r - p) mod N receives
    the partial of the sub-tree rooted at position p + d from rank
    (r + d) mod N.  A leaf's partial is its raw input; any other partial is
    the accumulation buffer it filled, which it gives up when sending.  The
    receiver adds the partial to its own accumulation buffer for tree c,
    starting it from its own input at its first receive, or, when c is its own
    chunk (p == 0), to its receive buffer.  Adds are single float32 roundings
    (int32 wraps); bfloat16 partials are carried in float32 and the receive
    buffer is rounded to bfloat16 once, after the last receive.

    `steps`, if given, replaces schedule(N, t, order) as the all-gather steps
    whose reversal is executed (checked the same way).
    """
    inputs = np.asarray(inputs)
    N = inputs.shape[0]
    if N == 1:
        return inputs[0].copy(), {"steps": 0, "chunks_per_step": [], "peak_per_dim": {}}
    root = [None] * N   # rank -> its own chunk's running sum
    acc = [dict() for _ in range(N)]  # rank -> {(d, chunk): partial}
    peak = {}
    steps = list(reversed(schedule(N, t, order) if steps is None else steps))
    for d, P in steps:
        arriving = []
        for r in range(N):
            for p in P:
                c = tree_of(r, p, N)
                child = peer_of(r, d, N)
                cpos = p + d
                leaf = children(N, cpos, d) == 0
                key = (d, c)  # the child's buffer for the dimension it sends on
                if leaf:
                    if key in acc[child]:
                        raise AssertionError("leaf holds an accumulation buffer")
                    partial = _widen(inputs[child, c], dtype)
                else:
                    if key not in acc[child]:
                        raise AssertionError(f"rank {child} sends a partial it never built")
                    partial = acc[child].pop(key)
                arriving.append((r, p, c, partial))
        for r, p, c, partial in arriving:
            if p == 0:
                own = root[r] if root[r] is not None else _widen(inputs[r, c], dtype)
                root[r] = _add(own, partial, dtype)
            else:
                key = (lowbit(p), c)
                own = acc[r].get(key)
                if own is None:
                    own = _widen(inputs[r, c], dtype)
                acc[r][key] = _add(own, partial, dtype)
        for r in range(N):
            held = {}
            for dd, _ in acc[r]:
                held[dd] = held.get(dd, 0) + 1
            for dd, n in held.items():
                peak[dd] = max(peak.get(dd, 0), n)
    if any(acc[r] for r in range(N)):
        raise AssertionError("accumulation buffers not drained")
    out = np.empty((N,) + inputs.shape[2:], dtype=inputs.dtype)
    for r in range(N):
        if dtype == "int32":
            out[r] = root[r].view(np.int32)
        elif dtype == "float32":
            out[r] = root[r]
        else:
            out[r] = f32_to_bf16_bits(root[r])
    stats = {"steps": len(steps), "chunks_per_step": [len(P) for _, P in steps],
             "peak_per_dim": peak}
    return out, stats


# --------------------------------------------------------------------------
# Closed form of the reduce-scatter association (far-first linear order)
# --------------------------------------------------------------------------

def reversed_tree_sum(values, nranks: int, add):
    """The sum one root obtains with the far-first schedule, written from the
    tree itself rather than from the steps (section "Conversion to
    reduce-scatter operations": the trees are reversed, close dimensions come
    first, and each received partial is added to the receiver's buffer).

    values[q] is the contribution of tree position q (rank root + q).  The node
    at position lo that owns span w (its reach) first completes the half-span
    it keeps, then adds the partial of its child at lo + w/2, which owns the
    other half -- unless truncation removed that child (lo + w/2 >= N).  Close
    children therefore arrive first, and the association is
        S(lo, 1) = v[lo]
        S(lo, w) = S(lo, w/2)                        if lo + w/2 >= N
                 = add(S(lo, w/2), S(lo + w/2, w/2)) otherwise,
    evaluated at S(0, 2^L), L = ceil(log2 N).  It does not depend on how many
    sub-trees run in parallel (T) or on splitting a chunk into pieces.

    `add` is the receiver's addition: a float32 add (one rounding), a wrapping
    int32 add, or a symbolic one in the pins."""
    L = ceil_log2(nranks)

    def S(lo, w):
        if w == 1:
            return values[lo]
        left = S(lo, w // 2)
        if lo + w // 2 >= nranks:
            return left
        return add(left, S(lo + w // 2, w // 2))

    return S(0, 1 << L)


def reducescatter_closed_form(inputs: np.ndarray, dtype: str) -> np.ndarray:
    """Reduce-scatter through reversed_tree_sum, destination by destination.

    inputs: (N, N, m), inputs[x][R] = rank x's contribution to chunk R;
    returns (N, m) in the input dtype.  Tree position q of root R is rank
    (R + q) mod N (all-gather data moves from r to r + d, so the reversed
    partials move from r + d to r).  int32 adds wrap; float32 adds round once
    each; bfloat16 values are widened exactly, added in float32 and rounded to
    bfloat16 once at the end."""
    inputs = np.asarray(inputs)
    N = inputs.shape[0]
    out = np.empty((N,) + inputs.shape[2:], dtype=inputs.dtype)
    if dtype == "int32":
        add = lambda a, b: (a + b).astype(np.uint32)  # noqa: E731  (wraps)
    elif dtype in ("float32", "bfloat16"):
        add = lambda a, b: (a + b).astype(np.float32)  # noqa: E731
    else:
        raise ValueError(dtype)
    for R in range(N):
        v = [_widen(inputs[rank_at(R, q, N), R], dtype) for q in range(N)]
        total = reversed_tree_sum(v, N, add)
        if dtype == "int32":
            out[R] = np.asarray(total, dtype=np.uint32).view(np.int32)
        elif dtype == "float32":
            out[R] = total
        else:
            out[R] = f32_to_bf16_bits(np.asarray(total, dtype=np.float32))
    return out
