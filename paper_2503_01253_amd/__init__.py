"""MI355X-native vector-wise N:M sparse matrix multiplication (NM-SpMM,
arXiv 2503.01253): C = A * B with B pruned N:M along k in blocks of V columns
and stored compressed as (Bc, idx).

The compute lives in libnmspmm.so (hand-written gfx950 HIP kernels behind a
C ABI declared in include/nmspmm.h); this package is its ctypes binding.
"""
from .binding import (  # noqa: F401
    ACTS, EXPORTS, NMSPMM_ACT_GELU, NMSPMM_ACT_NONE, NMSPMM_ACT_RELU, NMSPMM_ERR_HIP,
    NMSPMM_ERR_INVALID_ARG, NMSPMM_ERR_SCRATCH, NMSPMM_ERR_UNSUPPORTED, NMSPMM_NOALLOC_SCRATCH_BYTES, NMSPMM_OK, NmSpmmError, lib,
    nmspmm_bc_elems, nmspmm_compress, nmspmm_compress_device, nmspmm_confusion, nmspmm_idx_bytes,
    nmspmm_kernel_name, nmspmm_kernel_name_ws, nmspmm_run, nmspmm_run_ex, nmspmm_run_noalloc, nmspmm_run_ptr, nmspmm_run_ws,
    nmspmm_status_string, nmspmm_validate_idx, nmspmm_workspace_bytes,
)
