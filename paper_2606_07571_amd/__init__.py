"""BiCache shared-prefix denoising step for diffusion LMs on MI355X (gfx950).

The computation lives in libbicache.so (hand-written HIP kernels behind a C
ABI, declared in include/bicache.h); this package is a thin ctypes binding
over it plus the seeded synthetic-input generators used by tests and bench.
"""
from ._lib import (BiCacheError, LIB_PATH, Model, build_depth_table, cosine_similarity,  # noqa: F401
                   cosine_similarity_noalloc,
                   depth_lookup, is_refresh_step, lib, prefix_key, request_prefix_attention,
                   shallow_depth, shared_prefix_attention)
