"""Tile-sparse 3D attention (forward and gradients) for MI355X (gfx950).

The hot path of Efficient-vDiT (arXiv 2502.06155): softmax attention in which
each query latent frame only attends to the key frames its frame-tile mask
keeps (diagonal plus k global reference frames), computed by hand-written HIP
kernels behind a C ABI (include/tile_attn.h). This package is the thin Python
binding of that ABI.
"""
from .api import (  # noqa: F401
    MASK_FORMS,
    TileAttnError,
    dense_attn,
    dense_attn_fwd,
    tile_attn,
    tile_attn_bwd,
    tile_attn_bwd_mmdit,
    tile_attn_compact,
    tile_attn_fwd,
    tile_attn_fwd_heads,
    tile_attn_fwd_heads_noalloc,
    tile_attn_fwd_mmdit,
    tile_attn_make_mask,
    tile_attn_plan,
    tile_attn_plan_cache_stats,
)
