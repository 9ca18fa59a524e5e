"""Closed forms written from the tree definition (not from the oracle), shared
by the oracle's pins and by GPU checks at sizes the oracle's executors cannot
reach.  Test infrastructure: nothing here calls the HIP library or the oracle.
"""

import numpy as np


def tree_sum(v, n):
    """Reversed binomial tree, nearest child first (section "Conversion to
    reduce-scatter operations"), written from the tree: the node at `lo`
    owning span w first sums its own half-span, then adds the partial of the
    child at lo + w/2 (absent if truncated).  float32 adds.  v[q] is the
    value of tree position q (a scalar or an array: the sum runs elementwise).
    """
    L = (n - 1).bit_length()

    def S(lo, w):
        if w == 1:
            return v[lo]
        left = S(lo, w // 2)
        if lo + w // 2 >= n:
            return left
        return (left + S(lo + w // 2, w // 2)).astype(np.float32)

    return S(0, 1 << L)
