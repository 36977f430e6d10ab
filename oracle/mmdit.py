"""The MM-DiT form of tile-sparse attention, written out from its definition
(oracle side).

Test infrastructure only; see the package docstring.

In an MM-DiT (the CogVideoX extension of Sec. 4.3 and App. E) the attention input
concatenates text tokens with the video tokens, and the sparse mask is applied to
the video-video part only. Reading used here (the paper does not spell out the
layout): the P text tokens come first, then the F * T video tokens frame-major, so
token s < P is text and token s >= P belongs to video frame (s - P) // T.

  * a text query attends to every token (text and video);
  * a query of video frame i attends to every text token and to the tokens of the
    video frames j with mask[i, j] != 0.

Softmax over those keys of scale * <q_s, k_t>, as in ``oracle.attention``; with
P = 0 this is exactly that function. ``attention_mmdit_lse`` gives the natural-log
log-sum-exp per query. Masks are F x F (shared) or H x F x F (one per head).
Arithmetic is float64.
"""
from __future__ import annotations

import numpy as np

from .attention import as_f64, head_mask


def text_tokens(P: int) -> np.ndarray:
    return np.arange(P)


def video_frame_tokens(j: int, T: int, P: int) -> np.ndarray:
    """Token indices of video frame j after the P text tokens."""
    return np.arange(P + j * T, P + (j + 1) * T)


def key_tokens(mask_h: np.ndarray, i, T: int, P: int) -> np.ndarray:
    """Keys of a query in video frame i, or of a text query (i = None)."""
    F = mask_h.shape[0]
    if i is None:
        return np.arange(P + F * T)
    parts = [text_tokens(P)] + [video_frame_tokens(j, T, P) for j in range(F) if mask_h[i, j]]
    return np.concatenate(parts)


def _query_groups(F: int, T: int, P: int):
    """(frame or None, query token indices) for the text block and every video frame."""
    groups = [(None, text_tokens(P))] if P else []
    return groups + [(i, video_frame_tokens(i, T, P)) for i in range(F)]


def _shape(q, T: int, P: int, mask):
    B, H, S, d = np.shape(q)
    F = (S - P) // T
    if P < 0 or F * T + P != S:
        raise ValueError("q must be [B, H, P + F*T, d]")
    if np.asarray(mask).shape not in ((F, F), (H, F, F)):
        raise ValueError("mask must be F x F or H x F x F")
    return B, H, S, d, F


def attention_mmdit(q, k, v, mask, T: int, P: int, scale: float) -> np.ndarray:
    """Full output [B, H, P + F*T, d], float64; rows with no key stay zero."""
    mask = np.asarray(mask)
    B, H, S, d, F = _shape(q, T, P, mask)
    out = np.zeros((B, H, S, d))
    for b in range(B):
        for h in range(H):
            qh, kh, vh = as_f64(q[b, h]), as_f64(k[b, h]), as_f64(v[b, h])
            mh = head_mask(mask, h)
            for i, rows in _query_groups(F, T, P):
                cols = key_tokens(mh, i, T, P)
                if cols.size == 0:
                    continue
                logits = scale * (qh[rows] @ kh[cols].T)
                w = np.exp(logits - logits.max(axis=-1, keepdims=True))
                out[b, h, rows] = (w @ vh[cols]) / w.sum(axis=-1, keepdims=True)
    return out


def attention_mmdit_rows(q, k, v, mask, T: int, P: int, scale: float, b_idx, h_idx, s_idx):
    """Output rows for the listed (b, h, s) triples, float64 [n, d]."""
    mask = np.asarray(mask)
    B, H, S, d, F = _shape(q, T, P, mask)
    out = np.zeros((len(s_idx), d))
    for n, (b, h, s) in enumerate(zip(b_idx, h_idx, s_idx)):
        i = None if s < P else (int(s) - P) // T
        cols = key_tokens(head_mask(mask, int(h)), i, T, P)
        if cols.size == 0:
            continue
        logits = scale * (as_f64(k[b, h, cols]) @ as_f64(q[b, h, s]))
        w = np.exp(logits - logits.max())
        out[n] = (w @ as_f64(v[b, h, cols])) / w.sum()
    return out


def attention_mmdit_lse(q, k, mask, T: int, P: int, scale: float) -> np.ndarray:
    """Natural-log log-sum-exp [B, H, P + F*T] of each query's scaled logits; -inf for
    queries with no key."""
    mask = np.asarray(mask)
    B, H, S, d, F = _shape(q, T, P, mask)
    lse = np.full((B, H, S), -np.inf)
    for b in range(B):
        for h in range(H):
            qh, kh = as_f64(q[b, h]), as_f64(k[b, h])
            mh = head_mask(mask, h)
            for i, rows in _query_groups(F, T, P):
                cols = key_tokens(mh, i, T, P)
                if cols.size == 0:
                    continue
                logits = scale * (qh[rows] @ kh[cols].T)
                m = logits.max(axis=-1, keepdims=True)
                lse[b, h, rows] = (m + np.log(np.exp(logits - m).sum(axis=-1, keepdims=True)))[:, 0]
    return lse
