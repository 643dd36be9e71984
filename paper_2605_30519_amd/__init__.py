"""OmniMem memory-retrieval attention (arXiv 2605.30519) on AMD MI355X.

The compute path is libomnimem.so (hand-written HIP for gfx950, C ABI in
include/omnimem.h); ``omnimem`` is its thin ctypes binding and ``synth`` the
seeded synthetic-input generator.  Importing this package loads nothing: the
library is opened on the first call.
"""
from .omnimem import (  # noqa: F401
    EXPORTED,
    CompressedCache,
    LruOffload,
    OmniMemError,
    SCORE_LOGIT,
    SCORE_PROB,
    PagedKVCache,
    Selection,
    lib,
    library_path,
    omnimem_awe_active,
    omnimem_blocks_per_chunk,
    omnimem_cmp_attn,
    omnimem_compress_chunk,
    omnimem_dense_attn,
    omnimem_gated_combine,
    omnimem_select,
    omnimem_select_compressed,
    omnimem_select_noalloc,
    omnimem_select_workspace_bytes,
    omnimem_sparse_attn,
    omnimem_status_string,
    omnimem_union_gather_attn,
    omnimem_union_workspace_bytes,
    select_params,
    omnimem_numa_bind,
    omnimem_selected_chunks,
)
