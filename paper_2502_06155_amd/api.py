"""Python binding of the C ABI in include/tile_attn.h (argument marshalling only).

Every function forwards to the HIP library; all attention arithmetic runs in
the gfx950 kernels. PyTorch is used only to read device pointers and the
current stream of tensors handed in by the caller.
"""
from __future__ import annotations

import ctypes

import numpy as np

from ._lib import lib

TA_OK = 0
MASK_FORMS = {"col": 0, "sym": 1, "dense": 2}


class TileAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        text = lib.tile_attn_status_string(status).decode()
        detail = lib.tile_attn_last_error().decode()
        super().__init__(f"{where}: {text} ({status}): {detail}")


def _check(status: int, where: str) -> None:
    if status != TA_OK:
        raise TileAttnError(status, where)


def _ptr(x) -> int | None:
    """Device address of a torch tensor, or an integer address as given."""
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _stream(stream) -> int | None:
    if stream is None:
        return None
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream
    return int(stream)


def _mask_bytes(tile_mask, F: int) -> np.ndarray:
    m = np.ascontiguousarray(np.asarray(tile_mask), dtype=np.uint8)
    if m.size != F * F:
        raise ValueError(f"tile_mask must hold F*F = {F * F} entries, got {m.size}")
    return m


def tile_attn_fwd(q, k, v, out, B: int, H: int, F: int, T: int, d: int, tile_mask,
                  scale: float, stream=None) -> None:
    """tile_attn_fwd of the C ABI. q, k, v, out: device tensors or addresses."""
    m = _mask_bytes(tile_mask, F)
    _check(lib.tile_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, F, T, d,
                             m.ctypes.data, float(scale), _stream(stream)), "tile_attn_fwd")


def tile_attn_fwd_heads(q, k, v, out, B: int, H: int, F: int, T: int, d: int, tile_masks,
                        scale: float, lse=None, stream=None) -> None:
    """tile_attn_fwd_heads of the C ABI: tile_masks is F x F (shared) or H x F x F (one
    per head); lse is an optional fp32 [B, H, F*T] device tensor or address."""
    m = np.ascontiguousarray(np.asarray(tile_masks), dtype=np.uint8)
    if m.size % (F * F):
        raise ValueError("tile_masks must hold n_masks * F * F entries")
    n_masks = m.size // (F * F)
    _check(lib.tile_attn_fwd_heads(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, F, T, d,
                                   m.ctypes.data, n_masks, float(scale), _ptr(lse),
                                   _stream(stream)), "tile_attn_fwd_heads")


def tile_attn_fwd_heads_noalloc(q, k, v, out, B: int, H: int, F: int, T: int, d: int, tile_masks,
                                scale: float, lse=None, stream=None) -> None:
    """tile_attn_fwd_heads_noalloc of the C ABI: tile_attn_fwd_heads without any device
    allocation (plan and partials in the library's static per-GPU scratch array)."""
    m = np.ascontiguousarray(np.asarray(tile_masks), dtype=np.uint8)
    if m.size % (F * F):
        raise ValueError("tile_masks must hold n_masks * F * F entries")
    n_masks = m.size // (F * F)
    _check(lib.tile_attn_fwd_heads_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, F, T, d,
                                           m.ctypes.data, n_masks, float(scale), _ptr(lse),
                                           _stream(stream)), "tile_attn_fwd_heads_noalloc")


def tile_attn_fwd_mmdit(q, k, v, out, B: int, H: int, F: int, T: int, P: int, d: int,
                        tile_masks, scale: float, lse=None, stream=None) -> None:
    """tile_attn_fwd_mmdit of the C ABI: P text tokens before the F*T video tokens
    ([B, H, P + F*T, d]); tile_masks (F x F or H x F x F) cover the video part only."""
    m = np.ascontiguousarray(np.asarray(tile_masks), dtype=np.uint8)
    if m.size % (F * F):
        raise ValueError("tile_masks must hold n_masks * F * F entries")
    n_masks = m.size // (F * F)
    _check(lib.tile_attn_fwd_mmdit(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, F, T, P, d,
                                   m.ctypes.data, n_masks, float(scale), _ptr(lse),
                                   _stream(stream)), "tile_attn_fwd_mmdit")


def tile_attn_bwd(q, k, v, out, dout, lse, dq, dk, dv, B: int, H: int, F: int, T: int,
                  d: int, tile_masks, scale: float, stream=None) -> None:
    """tile_attn_bwd of the C ABI: gradients dq, dk, dv (bf16 [B, H, F*T, d]) from the
    forward's out and lse (fp32 [B, H, F*T]) and dout; tile_masks as for
    tile_attn_fwd_heads."""
    m = np.ascontiguousarray(np.asarray(tile_masks), dtype=np.uint8)
    if m.size % (F * F):
        raise ValueError("tile_masks must hold n_masks * F * F entries")
    n_masks = m.size // (F * F)
    _check(lib.tile_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
                             _ptr(dq), _ptr(dk), _ptr(dv), B, H, F, T, d, m.ctypes.data,
                             n_masks, float(scale), _stream(stream)), "tile_attn_bwd")


def tile_attn_bwd_mmdit(q, k, v, out, dout, lse, dq, dk, dv, B: int, H: int, F: int, T: int,
                        P: int, d: int, tile_masks, scale: float, stream=None) -> None:
    """tile_attn_bwd_mmdit of the C ABI: gradients of the MM-DiT form ([B, H, P + F*T, d],
    text first) from tile_attn_fwd_mmdit's out and lse."""
    m = np.ascontiguousarray(np.asarray(tile_masks), dtype=np.uint8)
    if m.size % (F * F):
        raise ValueError("tile_masks must hold n_masks * F * F entries")
    n_masks = m.size // (F * F)
    _check(lib.tile_attn_bwd_mmdit(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
                                   _ptr(dq), _ptr(dk), _ptr(dv), B, H, F, T, P, d, m.ctypes.data,
                                   n_masks, float(scale), _stream(stream)), "tile_attn_bwd_mmdit")


def dense_attn_fwd(q, k, v, out, B: int, H: int, F: int, T: int, d: int, scale: float,
                   stream=None) -> None:
    """dense_attn_fwd of the C ABI: every tile kept."""
    _check(lib.dense_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), B, H, F, T, d,
                              float(scale), _stream(stream)), "dense_attn_fwd")


def tile_attn_make_mask(F: int, k: int, form: str | int = "col") -> np.ndarray:
    """k:(F-k) mask as an F x F uint8 array (tile_attn_make_mask of the C ABI)."""
    f = MASK_FORMS[form] if isinstance(form, str) else int(form)
    out = np.zeros((F, F), dtype=np.uint8) if F >= 1 else np.zeros(1, dtype=np.uint8)
    _check(lib.tile_attn_make_mask(F, k, f, out.ctypes.data), "tile_attn_make_mask")
    return out


def tile_attn_compact(tile_mask):
    """Kept-tile list of a mask: (row_ptr int32[F+1], cols uint16[nnz], order uint16[F])."""
    m = np.asarray(tile_mask)
    F = m.shape[0]
    m = _mask_bytes(m, F)
    row_ptr = np.zeros(F + 1, dtype=np.int32)
    cols = np.zeros(F * F, dtype=np.uint16)
    order = np.zeros(F, dtype=np.uint16)
    nnz = ctypes.c_int(0)
    _check(lib.tile_attn_compact(m.ctypes.data, F, row_ptr.ctypes.data, cols.ctypes.data,
                                 order.ctypes.data, ctypes.byref(nnz)), "tile_attn_compact")
    return row_ptr, cols[: nnz.value].copy(), order


def tile_attn_plan(tile_mask):
    """Work plan of a mask: (items int32[n, 4] = frame, first kept entry, count, slot;
    number of partial slots)."""
    m = np.asarray(tile_mask)
    F = m.shape[0]
    m = _mask_bytes(m, F)
    cap = 33 * F
    items = np.zeros(4 * cap, dtype=np.int32)
    n_items, n_slots = ctypes.c_int(0), ctypes.c_int(0)
    _check(lib.tile_attn_plan(m.ctypes.data, F, items.ctypes.data, cap, ctypes.byref(n_items),
                              ctypes.byref(n_slots)), "tile_attn_plan")
    return items[: 4 * n_items.value].reshape(-1, 4).copy(), n_slots.value


def tile_attn_plan_cache_stats():
    """(live, retired): cached device plans and evicted ones still waiting for their
    kernels to finish (tile_attn_plan_cache_stats of the C ABI)."""
    live, retired = ctypes.c_int(0), ctypes.c_int(0)
    _check(lib.tile_attn_plan_cache_stats(ctypes.byref(live), ctypes.byref(retired)),
           "tile_attn_plan_cache_stats")
    return live.value, retired.value


def _shape_of(q, T: int):
    if q.dim() != 4:
        raise ValueError("expected [B, H, S, d] tensors")
    B, H, S, d = q.shape
    if S % T:
        raise ValueError(f"S = {S} is not a multiple of T = {T}")
    return B, H, S // T, d


def _check_tensors(q, *others):
    """q, k, v, out of the torch wrappers: the same [B, H, S, d] shape, contiguous
    bfloat16 on one GPU. Checked before anything is launched: the kernels read and
    write B*H*S*d elements of every tensor."""
    import torch

    for t in others:
        if tuple(t.shape) != tuple(q.shape):
            raise ValueError(f"k, v and out must have q's shape {tuple(q.shape)}, got {tuple(t.shape)}")
    for t in (q, *others):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must be contiguous bfloat16 on a GPU")
        if t.device != q.device:
            raise ValueError(f"every tensor must be on q's device {q.device}, got {t.device}")


def tile_attn(q, k, v, tile_mask, T: int, scale: float | None = None, out=None):
    """Torch convenience wrapper: [B, H, F*T, d] bf16 tensors on the current stream."""
    import torch

    B, H, F, d = _shape_of(q, T)
    if out is None:
        out = torch.empty_like(q)
    _check_tensors(q, k, v, out)
    if scale is None:
        scale = d ** -0.5
    tile_attn_fwd(q, k, v, out, B, H, F, T, d, tile_mask, scale,
                  torch.cuda.current_stream(q.device))
    return out


def dense_attn(q, k, v, T: int, scale: float | None = None, out=None):
    """Torch convenience wrapper of the dense control."""
    import torch

    B, H, F, d = _shape_of(q, T)
    if out is None:
        out = torch.empty_like(q)
    _check_tensors(q, k, v, out)
    if scale is None:
        scale = d ** -0.5
    dense_attn_fwd(q, k, v, out, B, H, F, T, d, scale, torch.cuda.current_stream(q.device))
    return out
