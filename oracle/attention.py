"""Tile-sparse 3D attention, written out from its definition (oracle side).

Test infrastructure only; see the package docstring.

Definition (Sec. 3.1 and Sec. 3.3 of the paper; the kernel-only benchmark of
Sec. 4.2.1 takes query, key, value and mask and returns the attention output;
App. B skips the masked blocks without materialising the mask):

The sequence of S = F * T tokens is flattened frame-major (Sec. 4.1), so token
s is in latent frame s // T. For a query token s of frame i, the kept keys are
the tokens of every key frame j with mask[i, j] != 0. With
logit_t = scale * <q_s, k_t> over the kept keys t,

    out_s = sum_t softmax(logit)_t * v_t,

and out_s = 0 when frame i keeps no key frame. The result is exact up to
rounding: a block-sparse kernel only avoids computing tiles whose weights are
absent from this sum.

A mask argument is either one F x F mask shared by all heads or an H x F x F
stack with one mask per head (the per-head patterns of the layer-wise search of
Sec. 3.3 and Alg. 1). ``attention_lse`` gives, per query token, the natural-log
log-sum-exp of its scaled logits over the kept keys, log sum_t exp(logit_t), and
-inf when its frame keeps nothing.

Arithmetic is float64. Inputs are bf16 bit patterns (uint16) widened exactly,
or float arrays used as given.
"""
from __future__ import annotations

import numpy as np


def as_f64(x: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) exactly to float64; pass floats through."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def kept_frames(mask: np.ndarray, i: int) -> list[int]:
    """Key frames kept by query frame i: the nonzero entries of mask row i."""
    return [j for j in range(mask.shape[1]) if mask[i, j]]


def frame_tokens(j: int, T: int) -> np.ndarray:
    """Token indices of latent frame j in the frame-major sequence."""
    return np.arange(j * T, (j + 1) * T)


def _softmax_rows_times_v(logits: np.ndarray, vk: np.ndarray) -> np.ndarray:
    """Row softmax of ``logits`` (two passes: max, then exp-sum) applied to vk."""
    m = logits.max(axis=-1, keepdims=True)
    w = np.exp(logits - m)
    z = w.sum(axis=-1, keepdims=True)
    return (w @ vk) / z


def head_mask(mask, h: int) -> np.ndarray:
    """The F x F mask of head h: the shared mask, or entry h of a per-head stack."""
    mask = np.asarray(mask)
    return mask if mask.ndim == 2 else mask[h]


def _check_mask(mask, H: int, F: int) -> None:
    if mask.shape not in ((F, F), (H, F, F)):
        raise ValueError("mask must be F x F or H x F x F")


def attention(q, k, v, mask, T: int, scale: float) -> np.ndarray:
    """Full output [B, H, S, d] of tile-sparse attention, float64."""
    mask = np.asarray(mask)
    B, H, S, d = np.shape(q)
    F = S // T
    if F * T != S:
        raise ValueError("q must be [B, H, F*T, d]")
    _check_mask(mask, H, F)
    out = np.zeros((B, H, S, d), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            qh, kh, vh = as_f64(q[b, h]), as_f64(k[b, h]), as_f64(v[b, h])
            mh = head_mask(mask, h)
            for i in range(F):
                kept = kept_frames(mh, i)
                if not kept:
                    continue  # no kept tile: the rows stay zero
                rows = frame_tokens(i, T)
                cols = np.concatenate([frame_tokens(j, T) for j in kept])
                logits = scale * (qh[rows] @ kh[cols].T)
                out[b, h, rows] = _softmax_rows_times_v(logits, vh[cols])
    return out


def attention_rows(q, k, v, mask, T: int, scale: float, b_idx, h_idx, s_idx) -> np.ndarray:
    """Output rows out[b, h, s, :] for the listed (b, h, s) triples, float64 [n, d].

    Same definition as ``attention``; only the requested rows are computed, so
    sampled checks at full size stay cheap.
    """
    mask = np.asarray(mask)
    B, H, S, d = np.shape(q)
    F = S // T
    b_idx, h_idx, s_idx = (np.asarray(a, dtype=np.int64) for a in (b_idx, h_idx, s_idx))
    out = np.zeros((len(s_idx), d), dtype=np.float64)
    groups: dict = {}
    for n, (b, h, s) in enumerate(zip(b_idx, h_idx, s_idx)):
        groups.setdefault((int(b), int(h), int(s) // T), []).append(n)
    _check_mask(mask, H, F)
    for (b, h, i), members in groups.items():
        kept = kept_frames(head_mask(mask, h), i)
        if not kept:
            continue
        cols = np.concatenate([frame_tokens(j, T) for j in kept])
        kh = as_f64(k[b, h, cols])
        vh = as_f64(v[b, h, cols])
        qs = as_f64(q[b, h, s_idx[members]])
        logits = scale * (qs @ kh.T)
        out[members] = _softmax_rows_times_v(logits, vh)
    return out


def attention_lse(q, k, mask, T: int, scale: float) -> np.ndarray:
    """Log-sum-exp [B, H, S] of the scaled logits over each query's kept keys,
    natural log, float64; -inf for query frames that keep nothing."""
    mask = np.asarray(mask)
    B, H, S, d = np.shape(q)
    F = S // T
    if F * T != S:
        raise ValueError("q must be [B, H, F*T, d]")
    _check_mask(mask, H, F)
    lse = np.full((B, H, S), -np.inf)
    for b in range(B):
        for h in range(H):
            qh, kh = as_f64(q[b, h]), as_f64(k[b, h])
            mh = head_mask(mask, h)
            for i in range(F):
                kept = kept_frames(mh, i)
                if not kept:
                    continue
                rows = frame_tokens(i, T)
                cols = np.concatenate([frame_tokens(j, T) for j in kept])
                logits = scale * (qh[rows] @ kh[cols].T)
                m = logits.max(axis=-1, keepdims=True)
                lse[b, h, rows] = (m + np.log(np.exp(logits - m).sum(axis=-1, keepdims=True)))[:, 0]
    return lse
