"""ctypes handle on libtileattn.so (the gfx950 HIP library).

There is no fallback: if the library is missing the import fails with a clear
message, so no caller can silently run something other than the HIP kernels.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtileattn.so")

EXPORTS = (
    "tile_attn_fwd",
    "tile_attn_fwd_heads",
    "tile_attn_fwd_heads_noalloc",
    "tile_attn_fwd_mmdit",
    "tile_attn_bwd",
    "tile_attn_bwd_mmdit",
    "dense_attn_fwd",
    "tile_attn_make_mask",
    "tile_attn_compact",
    "tile_attn_plan",
    "tile_attn_plan_cache_stats",
    "tile_attn_status_string",
    "tile_attn_last_error",
)


def _bind_to_torch_runtime() -> None:
    """Load torch first when it is installed.

    PyTorch ships its own libamdhip64 (soname libamdhip64.so.7). Loading torch
    before this library makes the dynamic linker resolve our libamdhip64.so.7
    dependency to that same, already loaded runtime, so the process holds one
    HIP runtime and the pointers and streams torch hands us are valid here.
    Loading this library first would pull in a second runtime from /opt/rocm,
    and two HSA runtimes in one process cannot share the GPU.
    """
    try:
        import torch  # noqa: F401
    except ImportError:
        pass


def _load() -> ctypes.CDLL:
    _bind_to_torch_runtime()
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(LIB_PATH)
    vp, ci, cf = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    lib.tile_attn_fwd.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, vp, cf, vp]
    lib.tile_attn_fwd.restype = ci
    lib.tile_attn_fwd_heads.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, vp, ci, cf, vp, vp]
    lib.tile_attn_fwd_heads.restype = ci
    lib.tile_attn_fwd_heads_noalloc.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, vp, ci, cf, vp, vp]
    lib.tile_attn_fwd_heads_noalloc.restype = ci
    lib.tile_attn_fwd_mmdit.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, vp, ci, cf, vp, vp]
    lib.tile_attn_fwd_mmdit.restype = ci
    lib.tile_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, vp, ci,
                                  cf, vp]
    lib.tile_attn_bwd.restype = ci
    lib.tile_attn_bwd_mmdit.argtypes = [vp] * 9 + [ci] * 6 + [vp, ci, cf, vp]
    lib.tile_attn_bwd_mmdit.restype = ci
    lib.dense_attn_fwd.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, vp]
    lib.dense_attn_fwd.restype = ci
    lib.tile_attn_make_mask.argtypes = [ci, ci, ci, vp]
    lib.tile_attn_make_mask.restype = ci
    lib.tile_attn_compact.argtypes = [vp, ci, vp, vp, vp, ctypes.POINTER(ci)]
    lib.tile_attn_compact.restype = ci
    lib.tile_attn_plan.argtypes = [vp, ci, vp, ci, ctypes.POINTER(ci), ctypes.POINTER(ci)]
    lib.tile_attn_plan.restype = ci
    lib.tile_attn_plan_cache_stats.argtypes = [ctypes.POINTER(ci), ctypes.POINTER(ci)]
    lib.tile_attn_plan_cache_stats.restype = ci
    lib.tile_attn_status_string.argtypes = [ci]
    lib.tile_attn_status_string.restype = ctypes.c_char_p
    lib.tile_attn_last_error.argtypes = []
    lib.tile_attn_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()
