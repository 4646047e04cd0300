"""Shifted Non-Local Search for AMD MI355X (gfx950).

The computation lives in libsnls.so (hand-written HIP kernels behind the C
ABI of include/snls.h); ``snls`` is its thin ctypes binding.
"""
from .snls import (  # noqa: F401
    SNLS_DIST_L2, SNLS_DIST_PROD, SNLS_MAX_K, SNLS_OP_AGGREGATE, SNLS_OP_BACKWARD, SNLS_OP_SEARCH, SnlsError,
    load_library, snls_abi_version, snls_aggregate, snls_backward, snls_search, snls_status_string, snls_topk,
    snls_workspace_size,
)
