"""Reference oracle for the ValueDiff eviction pass (TEST INFRASTRUCTURE ONLY).

Plain fp64 C (``vdref.c``) behind ctypes.  Only ``tests/``, the smoke check and
the CPU-baseline leg of the benchmark may import this package; the product
path (``paper_2609_23314_amd``) never does.  See ``vdref.c`` for the passages
of the paper each step follows and for the readings taken where the paper is
silent.
"""
from .vdref import (  # noqa: F401
    BF16, F32, L2, DIR, NORM, VARIANTS,
    Oracle, decode_elems, mean, score, select_topn, compact, evict_step, geometry, attention, load,
)
