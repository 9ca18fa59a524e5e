"""PAT (Parallel Aggregated Trees) all-gather and reduce-scatter on one MI355X.

The collectives run in ``libpat.so`` (HIP kernels for gfx950, C-ABI in
``include/pat.h``); ``pat`` is its thin ctypes binding.
"""

from . import pat  # noqa: F401
