"""ValueDiff eviction pass on MI355X (gfx950).

The pass (mean of the cached value vectors, per-token score, top-N keep,
slot-reuse gather of K and V) runs in hand-written HIP kernels behind the C ABI
of ``include/vd.h``; ``vd`` is its Python binding, ``driver`` runs block
prompt processing and decode on top of it, ``synth`` makes seeded synthetic
caches.  The library is loaded on first use and must have been built
(``python -m paper_2609_23314_amd.build``).
"""
from .vd import (  # noqa: F401
    LIB_PATH, MAX_CAPACITY, VARIANTS, VdError, cache_desc, load,
    vd_compact, vd_evict_step, vd_evict_step_workspace_size, vd_score, vd_select_topn,
)
