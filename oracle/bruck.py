"""Nearest-dimension-first Bruck all-gather, as the paper enumerates it.

Test infrastructure only (see the package docstring).

Section "Binomial-tree based algorithms" describes the algorithm step by step:
at dimension n every rank sends the data it holds for ranks
myrank-(2^n - 1) .. myrank to myrank + 2^n, and receives the data for ranks
myrank-(2^(n+1) - 1) .. myrank - 2^n from myrank - 2^n.  The dimension n is
the power of two a rank communicates with.

For a rank count that is not a power of two the last dimension only has to
complete the set: a rank still missing N - 2^n chunks receives exactly those
(the truncation the same section applies to the binomial trees).  This module
is used only to cross-check ``definitions.allgather`` and ``pat`` on tiny N.
"""


def steps(nranks: int):
    """Yield (n, d, payload) per step; payload(r) lists the chunk ids rank r
    sends to rank r + d, nearest first (its own chunk first)."""
    n, d = 0, 1
    while d < nranks:
        width = min(d, nranks - d)  # chunks still missing at the receiver

        def payload(r, d=d, width=width):
            return [(r - j) % nranks for j in range(width)]

        yield n, d, payload
        n, d = n + 1, 2 * d


def allgather(chunks):
    """Run the step description on per-rank data.

    ``chunks[x]`` is rank x's own data (any object).  Returns (held, log):
    ``held[r]`` maps chunk id -> data for every chunk rank r ends with, and
    ``log`` lists, per step, (d, {sender: [chunk ids sent]}).
    """
    nranks = len(chunks)
    held = [{x: chunks[x]} for x in range(nranks)]
    log = []
    for _, d, payload in steps(nranks):
        messages = []
        sent = {}
        for r in range(nranks):
            ids = payload(r)
            for c in ids:
                if c not in held[r]:
                    raise AssertionError(f"rank {r} sends chunk {c} it does not hold")
            messages.append(((r + d) % nranks, {c: held[r][c] for c in ids}))
            sent[r] = ids
        for dst, data in messages:
            for c, v in data.items():
                if c in held[dst]:
                    raise AssertionError(f"rank {dst} receives chunk {c} twice")
                held[dst][c] = v
        log.append((d, sent))
    return held, log
