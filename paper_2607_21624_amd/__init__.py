"""Layout-copy-free attention forward/backward for MI355X (gfx950).

Multi-head (and grouped-query) attention forward and backward run directly on
token-major [B, S, H*d] activations through hand-written HIP kernels behind a
C ABI (include/fbl.h, libfbl.so).  This package is the Python binding:
argument marshalling only, torch for device memory and streams.
"""
from .fbl import (  # noqa: F401
    EXPORTED, FBL_BF16, FBL_BWD_ALL, FBL_BWD_KV, FBL_BWD_PREP, FBL_BWD_Q, FBL_F32, FBL_MASK_CAUSAL, FBL_MASK_KEY_PADDING, FblError, LIB, LIB_PATH, Layout, Mask,
    attn_bwd, attn_bwd_packed, attn_fwd, attn_fwd_packed, fbl_attn_bwd_raw, fbl_attn_bwd_workspace, fbl_attn_bwd_workspace_min, fbl_attn_fwd_raw,
    fbl_layout_desc, fbl_layout_packed_qkv, fbl_proj_raw, proj, FBL_PROJ_FWD, FBL_PROJ_BWD_DATA, FBL_PROJ_BWD_WEIGHT,
    FBL_GEMM_TILE_AUTO, FBL_GEMM_TILE_128x128, FBL_GEMM_TILE_128x64, FBL_GEMM_TILE_64x128, FBL_GEMM_TILE_64x64,
    FBL_TUNE_TIME, FBL_TUNE_GFLOPS_X_MEMEFF, gemm_tiles, proj_candidates, proj_tune, proj_tuned_tile, proj_auto_tile, proj_tune_reset,
    fbl_layout_desc_status, fbl_layout_map_device, fbl_layout_offset, layout_of, status_str,
    NOALLOC_SCRATCH_BYTES, attn_bwd_noalloc, fbl_attn_bwd_noalloc_raw,
    FBL_ATTN_FWD, FBL_ATTN_BWD_KV, FBL_ATTN_BWD_DQ, FBL_ATTN_TILE_AUTO, attn_tiles, attn_candidates, attn_auto_tiles, attn_bwd_launches,
    attn_tune, attn_tuned_tile, attn_tune_reset,
)
