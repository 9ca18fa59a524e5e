"""CPU oracle for PAT all-gather and reduce-scatter.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code, headers,
tables or helpers with the HIP library; the only thing both sides consume is
the seeded input generator in ``synth/``, which holds none of the method's
arithmetic.

Contents (all plain, slow and written to be checked against the paper by eye):

* ``definitions`` -- what the two collectives compute, by definition
  (all-gather = concatenation; reduce-scatter = elementwise sum, accumulated
  in fp64 / int64).  Section "All-gather and reduce-scatter algorithms".
* ``bruck``       -- the nearest-dimension-first Bruck all-gather exactly as
  the enumerated description in section "Binomial-tree based algorithms"
  states it.  Used only to cross-check the other two modules on tiny N.
* ``pat``         -- the PAT schedule (shifted binomial trees, farthest
  dimension first, truncation for non-power-of-two rank counts, aggregation
  limited to T parallel sub-trees with a far-first linear schedule inside
  them) and step-by-step executors for all-gather and for reduce-scatter
  (reversed trees, close dimensions first, accumulation buffers).  Sections
  "The PAT algorithm" and "Conversion to reduce-scatter operations".

Parity status: every function here is pinned by tests in
``tests/test_oracle_pins.py``.  The reduce-scatter's float32 association is
pinned to the reversed-tree closed form written in the tests from the tree
definition, to its invariance across aggregation levels and to the pairwise
error bound; which association the paper intends is a reading (the paper
prints no values), listed with the others in the design notes, and the
tolerance check against the fp64 plain sum does not depend on it.
"""
