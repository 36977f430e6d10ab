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


def attention_backward_mmdit(q, k, v, dout, mask, T: int, P: int, scale: float):
    """Gradients (dq, dk, dv), float64 [B, H, P + F*T, d], of ``attention_mmdit`` for the
    upstream gradient dout: the chain rule through each query's softmax over its keys,
    dS = P (dP - delta) with dP = dO V^T and delta = <dO, out>; dq = scale dS K,
    dk = scale dS^T Q, dv = P^T dO (sums over the query-key pairs the form keeps)."""
    mask = np.asarray(mask)
    B, H, S, d, F = _shape(q, T, P, mask)
    dq, dk, dv = (np.zeros((B, H, S, d)) for _ in range(3))
    for b in range(B):
        for h in range(H):
            qh, kh, vh, gh = (as_f64(x[b, h]) for x in (q, k, v, dout))
            mh = head_mask(mask, h)
            for i, rows in _query_groups(F, T, P):
                cols = key_tokens(mh, i, T, P)
                if cols.size == 0:
                    continue
                logits = scale * (qh[rows] @ kh[cols].T)
                w = np.exp(logits - logits.max(axis=-1, keepdims=True))
                p = w / w.sum(axis=-1, keepdims=True)
                out = p @ vh[cols]
                ds = p * (gh[rows] @ vh[cols].T - (gh[rows] * out).sum(axis=-1, keepdims=True))
                dq[b, h, rows] += scale * (ds @ kh[cols])
                dk[b, h, cols] += scale * (ds.T @ qh[rows])
                dv[b, h, cols] += p.T @ gh[rows]
    return dq, dk, dv


def attention_backward_mmdit_rows(q, k, v, dout, mask, T: int, P: int, scale: float, bq, hq, sq,
                                  bk, hk, sk, chunk: int = 512):
    """``attention_backward_mmdit`` at chosen rows only: dq at query tokens (bq, hq, sq)
    and dk, dv at key tokens (bk, hk, sk), float64 [n, d]; a key's gradient sums over
    every query whose key set holds it, ``chunk`` query rows at a time."""
    mask = np.asarray(mask)
    B, H, S, d, F = _shape(q, T, P, mask)
    dq = np.zeros((len(sq), d))
    dk = np.zeros((len(sk), d))
    dv = np.zeros((len(sk), d))
    bq, hq, sq, bk, hk, sk = (np.asarray(x, dtype=np.int64) for x in (bq, hq, sq, bk, hk, sk))

    def terms(qh, kh, vh, gh, cols, rows):
        logits = scale * (qh[rows] @ kh[cols].T)
        w = np.exp(logits - logits.max(axis=-1, keepdims=True))
        p = w / w.sum(axis=-1, keepdims=True)
        delta = (gh[rows] * (p @ vh[cols])).sum(axis=-1)
        return p, delta

    heads = sorted(set(zip(bq.tolist(), hq.tolist())) | set(zip(bk.tolist(), hk.tolist())))
    for (b, h) in heads:
        qh, kh, vh, gh = (as_f64(x[b, h]) for x in (q, k, v, dout))
        mh = head_mask(mask, h)
        for n in np.nonzero((bq == b) & (hq == h))[0]:
            s = int(sq[n])
            cols = key_tokens(mh, None if s < P else (s - P) // T, T, P)
            p, delta = terms(qh, kh, vh, gh, cols, np.array([s]))
            ds = p * (gh[[s]] @ vh[cols].T - delta[:, None])
            dq[n] = scale * (ds @ kh[cols])[0]
        sel = np.nonzero((bk == b) & (hk == h))[0]
        if sel.size == 0:
            continue
        keys = sk[sel]
        for i, rows_all in _query_groups(F, T, P):
            cols = key_tokens(mh, i, T, P)
            hit = np.isin(keys, cols)
            if not hit.any():
                continue
            tsel, kidx = sel[hit], keys[hit]
            pos = {int(c): m for m, c in enumerate(cols)}
            at = np.array([pos[int(t)] for t in kidx])
            for r0 in range(0, len(rows_all), chunk):
                rows = rows_all[r0:r0 + chunk]
                p, delta = terms(qh, kh, vh, gh, cols, rows)
                p_t = p[:, at]
                ds_t = p_t * (gh[rows] @ vh[kidx].T - delta[:, None])
                dk[tsel] += scale * (ds_t.T @ qh[rows])
                dv[tsel] += p_t.T @ gh[rows]
    return dq, dk, dv
