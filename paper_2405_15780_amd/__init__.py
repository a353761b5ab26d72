"""Exact non-causal multi-head attention (forward and backward) for MI355X.

A thin ctypes binding over the C ABI in include/vitattn.h; it only marshals
arguments. Every step of the computation runs in the library's HIP kernels.
PyTorch is used for device memory and the current stream only. If the built
library is missing the import of a binding function raises: there is no
fallback path.
"""
from .binding import (  # noqa: F401
    LIB_PATH,
    VITATTN_BWD_ACCUMULATE_DQ,
    VITATTN_BWD_STORE_DS,
    VITATTN_NOALLOC_MAX_ROWS,
    Strides,
    VitattnError,
    agg_bwd,
    agg_fwd,
    bwd,
    bwd_dkdv,
    bwd_dkdv_ds,
    bwd_dq,
    bwd_dq_from_ds,
    bwd_noalloc,
    bwd_rowdot,
    fwd,
    library,
    merge,
    status_str,
    strides_of,
    ulysses_pack,
    ulysses_pack_out,
    ulysses_unpack,
    ulysses_unpack_out,
    version,
    workspace_bytes,
    workspace_bytes_kv,
)
from .autograd import attention  # noqa: F401,E402
