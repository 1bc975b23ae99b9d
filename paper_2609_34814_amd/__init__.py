"""MI355X (gfx950) block-sparse attention with cache-aware query-row reordering.

The compute path lives in libwavealign.so (hand-written HIP); this package only
marshals torch tensors into its C ABI (include/wavealign.h).
"""
from .api import (attn_vt_workspace_size, attn_workspace_size, build_permutation, check_perm, compact_mask,
                  default_skip_profile, fp64_probe, mask_producer_workspace_size, mask_stats, perm_workspace_size,
                  produce_block_mask, shape_of, sparse_attn, sparse_attn_csr, sparse_attn_vt, sparse_attn_vt_noalloc,
                  transpose_v, wave_size, xcc_probe)
from ._lib import WaError, load as load_library

__all__ = ["attn_vt_workspace_size", "attn_workspace_size", "build_permutation", "check_perm", "compact_mask",
           "default_skip_profile", "fp64_probe", "mask_producer_workspace_size", "mask_stats", "perm_workspace_size",
           "produce_block_mask", "shape_of", "sparse_attn", "sparse_attn_csr", "sparse_attn_vt",
           "sparse_attn_vt_noalloc", "transpose_v",
           "wave_size", "xcc_probe", "WaError", "load_library"]
