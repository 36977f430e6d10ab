"""Gradients of tile-sparse 3D attention, written out from their definition (oracle side).

Test infrastructure only; see the package docstring.

The forward output of query token s (Sec. 3.3; ``oracle.attention``) is
out_s = sum_t P_st v_t with P_st = softmax_t(scale * <q_s, k_t>) over the keys t
of the frames that s's frame keeps. Its gradients, for an upstream gradient dO,
follow from the chain rule through the softmax (the training of the sparse
student in Sec. 3.4 back-propagates through this operation):

    dP_st = <dO_s, v_t>
    dS_st = P_st * (dP_st - D_s),  D_s = sum_t P_st dP_st = <dO_s, out_s>
    dq_s  = scale * sum_t dS_st k_t
    dk_t  = scale * sum_s dS_st q_s
    dv_t  = sum_s P_st dO_s

with sums over kept pairs only. Keys of frames nobody keeps get zero gradient,
and so do queries of frames that keep nothing. A mask is F x F (shared by the
heads) or H x F x F (one per head). Arithmetic is float64.
"""
from __future__ import annotations

import numpy as np

from .attention import as_f64, frame_tokens, head_mask, kept_frames


def attention_backward(q, k, v, dout, mask, T: int, scale: float):
    """(dq, dk, dv), each float64 [B, H, S, d], for upstream gradient dout."""
    mask = np.asarray(mask)
    B, H, S, d = np.shape(q)
    F = S // T
    if F * T != S or mask.shape not in ((F, F), (H, F, F)):
        raise ValueError("q must be [B, H, F*T, d] and mask F x F or H x F x F")
    dq = np.zeros((B, H, S, d))
    dk = np.zeros((B, H, S, d))
    dv = np.zeros((B, H, S, d))
    for b in range(B):
        for h in range(H):
            qh, kh, vh, gh = (as_f64(x[b, h]) for x in (q, k, v, dout))
            mh = head_mask(mask, h)
            for i in range(F):
                kept = kept_frames(mh, i)
                if not kept:
                    continue
                rows = frame_tokens(i, T)
                cols = np.concatenate([frame_tokens(j, T) for j in kept])
                logits = scale * (qh[rows] @ kh[cols].T)
                w = np.exp(logits - logits.max(axis=-1, keepdims=True))
                p = w / w.sum(axis=-1, keepdims=True)
                out = p @ vh[cols]
                dp = gh[rows] @ vh[cols].T
                big_d = (gh[rows] * out).sum(axis=-1, keepdims=True)
                ds = p * (dp - big_d)
                dq[b, h, rows] += scale * (ds @ kh[cols])
                dk[b, h, cols] += scale * (ds.T @ qh[rows])
                dv[b, h, cols] += p.T @ gh[rows]
    return dq, dk, dv


def _row_terms(qh, kh, vh, gh, kept, rows, T, scale):
    """For query rows `rows` (token indices) whose frame keeps frames `kept`: the kept
    key tokens, P over them, and delta = <dO, out> per row."""
    cols = np.concatenate([frame_tokens(j, T) for j in kept])
    logits = scale * (qh[rows] @ kh[cols].T)
    w = np.exp(logits - logits.max(axis=-1, keepdims=True))
    p = w / w.sum(axis=-1, keepdims=True)
    out = p @ vh[cols]
    big_d = (gh[rows] * out).sum(axis=-1)
    return cols, p, big_d


def attention_backward_rows(q, k, v, dout, mask, T: int, scale: float, bq, hq, sq, bk, hk, sk,
                            chunk: int = 512):
    """The gradients of ``attention_backward`` at chosen rows only: dq at query tokens
    (bq[i], hq[i], sq[i]) and dk, dv at key tokens (bk[i], hk[i], sk[i]), each float64
    [n, d]. Same definitions, restricted: a key's gradient sums over every query token
    whose frame keeps the key's frame, taken ``chunk`` query rows at a time."""
    mask = np.asarray(mask)
    B, H, S, d = np.shape(q)
    F = S // T
    bq, hq, sq = (np.asarray(x, dtype=np.int64) for x in (bq, hq, sq))
    bk, hk, sk = (np.asarray(x, dtype=np.int64) for x in (bk, hk, sk))
    dq = np.zeros((len(sq), d))
    dk = np.zeros((len(sk), d))
    dv = np.zeros((len(sk), d))
    cache = {}

    def head(b, h):
        if (b, h) not in cache:
            cache.clear()
            cache[(b, h)] = tuple(as_f64(x[b, h]) for x in (q, k, v, dout))
        return cache[(b, h)]

    for (b, h) in sorted(set(zip(bq.tolist(), hq.tolist()))):
        qh, kh, vh, gh = head(b, h)
        mh = head_mask(mask, h)
        sel = np.nonzero((bq == b) & (hq == h))[0]
        for n in sel:
            s = int(sq[n])
            kept = kept_frames(mh, s // T)
            if not kept:
                continue
            cols, p, big_d = _row_terms(qh, kh, vh, gh, kept, np.array([s]), T, scale)
            ds = p * (gh[[s]] @ vh[cols].T - big_d[:, None])
            dq[n] = scale * (ds @ kh[cols])[0]

    for (b, h) in sorted(set(zip(bk.tolist(), hk.tolist()))):
        qh, kh, vh, gh = head(b, h)
        mh = head_mask(mask, h)
        sel = np.nonzero((bk == b) & (hk == h))[0]
        keys = sk[sel]
        for i in range(F):
            kept = kept_frames(mh, i)
            hit = np.array([mh[i][int(t) // T] != 0 for t in keys])
            if not hit.any():
                continue
            tsel, kidx = sel[hit], keys[hit]
            rows_all = frame_tokens(i, T)
            for r0 in range(0, T, chunk):
                rows = rows_all[r0:r0 + chunk]
                cols, p, big_d = _row_terms(qh, kh, vh, gh, kept, rows, T, scale)
                pos = {int(c): m for m, c in enumerate(cols)}
                at = np.array([pos[int(t)] for t in kidx])
                p_t = p[:, at]
                dp_t = gh[rows] @ vh[kidx].T
                ds_t = p_t * (dp_t - big_d[:, None])
                dk[tsel] += scale * (ds_t.T @ qh[rows])
                dv[tsel] += p_t.T @ gh[rows]
    return dq, dk, dv
