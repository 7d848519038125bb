"""HiSparse decode hot path on AMD Instinct MI355X (gfx950).

The compute lives in libhisparse.so (hand-written HIP kernels behind the C ABI of
include/hisparse.h); `hisparse` is its ctypes binding. `HiSparseCache` is a small convenience
owner of one handle.
"""
from .hisparse import (AttnDesc, CacheDesc, HisparseError, hisparse_cache_create,  # noqa: F401
                       hisparse_cache_destroy, hisparse_check_errors,
                       hisparse_decode_workspace_bytes, hisparse_fetch, hisparse_host_pool,
                       hisparse_layer_cache, hisparse_prefetch_layer, hisparse_read_plan,
                       hisparse_read_state, hisparse_reset, hisparse_resolve, hisparse_resolve_tables,
                       hisparse_sparse_decode, hisparse_sparse_decode_pool,
                       hisparse_status_string, hisparse_validate_attn, hisparse_validate_desc,
                       host_view, lib)
from .cache import HiSparseCache  # noqa: F401
