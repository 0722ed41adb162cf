"""MI355X (gfx950) implementation of the HSA forward pass of WorldAttention.

The computation lives in libhsa.so (C ABI in include/hsa.h, HIP kernels in
csrc/). ``hsa`` is its ctypes binding; ``layer`` holds device buffers of one
attention layer and calls the binding.
"""
from .hsa import (  # noqa: F401
    HSA_DTYPE_BF16,
    HSA_DTYPE_F32,
    HsaConfig,
    HsaError,
    HsaKvPool,
    HsaTier,
    LibraryNotBuilt,
    TAU_MAX,
    TAU_MIN,
    config,
    hsa_adaptive_workspace_size,
    hsa_block_count,
    hsa_block_select,
    hsa_chunk_select,
    hsa_forward_adaptive,
    hsa_forward_noalloc,
    hsa_forward_noalloc_bytes,
    hsa_forward_retrieval,
    hsa_retrieval_workspace_size,
    hsa_forward_linformer,
    hsa_linformer_compress,
    hsa_linformer_compress_workspace_size,
    hsa_linformer_workspace_size,
    hsa_sparse_attn_adaptive,
    hsa_forward,
    hsa_forward_selected,
    hsa_forward_workspace_size,
    hsa_cube_order,
    hsa_page_select,
    hsa_page_write,
    hsa_page_select_workspace_size,
    hsa_sparse_attn,
    hsa_sparse_attn_workspace_size,
    hsa_state_update,
    hsa_state_update_workspace_size,
    hsa_status_string,
    kv_pool,
    lib,
)
from .layer import HsaLayer  # noqa: F401
