"""Pins of the attention oracle against facts the mathematics fixes.

Each pin takes an implementation with the oracle's signature
``attn(q, k, v, mask, T, scale)`` (float64 arrays [B, H, F*T, d], F x F mask)
and raises AssertionError when it disagrees. None of them re-runs the oracle's
own formula: they compare against torch's CPU scaled_dot_product_attention
(a library routine), a pure-Python brute force without the max shift, closed
forms, and invariances of the definition (Sec. 3.3 of the paper).
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import torch

TOL = 1e-12


def _rand(rng, B, H, S, d, scale=1.0):
    return rng.standard_normal((B, H, S, d)) * scale


def _sdpa_masked(q, k, v, mask, T, scale):
    """Masked attention by torch SDPA with a token-level boolean mask; empty rows -> 0."""
    F = mask.shape[0]
    frame = np.arange(F * T) // T
    tok = np.asarray(mask, dtype=bool)[frame][:, frame]  # [S, S]
    qt, kt, vt = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    empty = ~tok.any(axis=1)
    tok_safe = tok.copy()
    tok_safe[empty, :] = True  # avoid all-masked rows inside SDPA
    out = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=torch.from_numpy(tok_safe), scale=scale
    ).numpy()
    out[:, :, empty, :] = 0.0
    return out


def pin_dense_matches_sdpa(attn):
    rng = np.random.default_rng(1)
    for (B, H, F, T, d) in [(1, 2, 3, 5, 8), (2, 1, 2, 7, 4), (1, 1, 1, 9, 16)]:
        q, k, v = (_rand(rng, B, H, F * T, d) for _ in range(3))
        scale = 1 / math.sqrt(d)
        ref = torch.nn.functional.scaled_dot_product_attention(
            *(torch.from_numpy(x) for x in (q, k, v)), scale=scale).numpy()
        got = attn(q, k, v, np.ones((F, F), np.uint8), T, scale)
        assert np.max(np.abs(got - ref)) < TOL, "dense mask differs from textbook attention"


def pin_all_small_masks_match_sdpa(attn):
    """Every one of the 2^(F*F) masks for F <= 3 against library attention."""
    rng = np.random.default_rng(2)
    for F, T, d in [(1, 4, 4), (2, 3, 4), (3, 2, 4)]:
        q, k, v = (_rand(rng, 1, 1, F * T, d) for _ in range(3))
        for bits in itertools.product((0, 1), repeat=F * F):
            mask = np.array(bits, dtype=np.uint8).reshape(F, F)
            got = attn(q, k, v, mask, T, 0.7)
            ref = _sdpa_masked(q, k, v, mask, T, 0.7)
            assert np.max(np.abs(got - ref)) < TOL, f"mask {bits} differs"


def pin_random_masks_match_sdpa(attn):
    rng = np.random.default_rng(3)
    for trial in range(6):
        F = int(rng.integers(2, 6))
        T = int(rng.choice([1, 3, 17]))
        d = int(rng.choice([4, 16]))
        B, H = 1 + trial % 2, 2
        mask = (rng.random((F, F)) < 0.5).astype(np.uint8)
        q, k, v = (_rand(rng, B, H, F * T, d) for _ in range(3))
        scale = float(rng.uniform(0.1, 1.5))
        got = attn(q, k, v, mask, T, scale)
        ref = _sdpa_masked(q, k, v, mask, T, scale)
        assert np.max(np.abs(got - ref)) < TOL


def pin_bruteforce(attn):
    """Pure-Python loops over tokens, normalising sum(exp) directly (no max shift)."""
    rng = np.random.default_rng(4)
    F, T, d = 3, 4, 3
    mask = np.array([[1, 0, 1], [0, 0, 0], [1, 1, 0]], dtype=np.uint8)
    q, k, v = (_rand(rng, 1, 1, F * T, d, 0.5) for _ in range(3))
    scale = 0.9
    got = attn(q, k, v, mask, T, scale)
    for s in range(F * T):
        kept = [t for t in range(F * T) if mask[s // T][t // T]]
        if not kept:
            expect = [0.0] * d
        else:
            w = {t: math.exp(scale * sum(q[0, 0, s, c] * k[0, 0, t, c] for c in range(d))) for t in kept}
            z = sum(w.values())
            expect = [sum(w[t] * v[0, 0, t, c] for t in kept) / z for c in range(d)]
        assert max(abs(got[0, 0, s, c] - expect[c]) for c in range(d)) < TOL, f"row {s}"


def pin_constant_values(attn):
    """Softmax weights sum to one: V constant per column reproduces the constant."""
    rng = np.random.default_rng(5)
    F, T, d = 4, 6, 8
    mask = (rng.random((F, F)) < 0.6).astype(np.uint8)
    mask[2, :] = 0
    q, k = (_rand(rng, 1, 2, F * T, d) for _ in range(2))
    c = rng.standard_normal(d)
    v = np.broadcast_to(c, (1, 2, F * T, d)).copy()
    got = attn(q, k, v, mask, T, 0.5)
    for s in range(F * T):
        expect = c if mask[s // T].any() else np.zeros(d)
        assert np.max(np.abs(got[0, :, s] - expect)) < TOL


def pin_uniform_weights(attn):
    """Q = 0 (or scale = 0) gives equal weights: the mean of V over the kept frames."""
    rng = np.random.default_rng(6)
    F, T, d = 4, 5, 6
    mask = np.array([[1, 1, 0, 0], [0, 1, 0, 1], [0, 0, 0, 0], [1, 1, 1, 1]], dtype=np.uint8)
    k, v = (_rand(rng, 1, 1, F * T, d) for _ in range(2))
    frame_mean = v[0, 0].reshape(F, T, d).mean(axis=1)
    for q, scale in [(np.zeros_like(k), 0.8), (_rand(rng, 1, 1, F * T, d), 0.0)]:
        got = attn(q, k, v, mask, T, scale)
        for i in range(F):
            kept = np.flatnonzero(mask[i])
            expect = frame_mean[kept].mean(axis=0) if len(kept) else np.zeros(d)
            assert np.max(np.abs(got[0, 0, i * T:(i + 1) * T] - expect)) < TOL


def pin_identical_frames(attn):
    """If every frame's K/V is the same copy, any mask with a kept tile per row equals
    attention over that one frame (repeating keys leaves softmax unchanged)."""
    rng = np.random.default_rng(7)
    F, T, d = 4, 6, 8
    k1, v1 = (_rand(rng, 1, 1, T, d) for _ in range(2))
    k, v = np.tile(k1, (1, 1, F, 1)), np.tile(v1, (1, 1, F, 1))
    q = _rand(rng, 1, 1, F * T, d)
    mask = np.eye(F, dtype=np.uint8)
    mask[:, 0] = 1
    mask[3, :] = 1
    got = attn(q, k, v, mask, T, 0.6)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k1), torch.from_numpy(v1), scale=0.6).numpy()
    assert np.max(np.abs(got - ref)) < TOL


def pin_key_frame_permutation(attn):
    """Relabelling key frames (K/V frames and mask columns together) changes nothing."""
    rng = np.random.default_rng(8)
    F, T, d = 5, 3, 4
    q, k, v = (_rand(rng, 1, 1, F * T, d) for _ in range(3))
    mask = (rng.random((F, F)) < 0.5).astype(np.uint8)
    mask[np.arange(F), np.arange(F)] = 1
    perm = rng.permutation(F)
    kp = k.reshape(1, 1, F, T, d)[:, :, perm].reshape(1, 1, F * T, d)
    vp = v.reshape(1, 1, F, T, d)[:, :, perm].reshape(1, 1, F * T, d)
    a = attn(q, k, v, mask, T, 0.8)
    b = attn(q, kp, vp, mask[:, perm], T, 0.8)
    assert np.max(np.abs(a - b)) < TOL


def pin_per_head_masks_match_sdpa(attn):
    """An H x F x F stack applies mask h to head h (torch SDPA with that head's token
    mask, head by head); a shared mask equals the stack of H copies."""
    rng = np.random.default_rng(9)
    B, H, F, T, d = 2, 3, 4, 3, 8
    q, k, v = (_rand(rng, B, H, F * T, d) for _ in range(3))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    masks[1, 2, :] = 0
    got = attn(q, k, v, masks, T, 0.6)
    for h in range(H):
        ref = _sdpa_masked(q[:, h:h + 1], k[:, h:h + 1], v[:, h:h + 1], masks[h], T, 0.6)
        assert np.max(np.abs(got[:, h:h + 1] - ref)) < TOL, f"head {h}"
    shared = attn(q, k, v, masks[0], T, 0.6)
    stacked = attn(q, k, v, np.stack([masks[0]] * H), T, 0.6)
    assert np.max(np.abs(shared - stacked)) < TOL


ALL_PINS = [
    pin_dense_matches_sdpa,
    pin_all_small_masks_match_sdpa,
    pin_random_masks_match_sdpa,
    pin_bruteforce,
    pin_constant_values,
    pin_uniform_weights,
    pin_identical_frames,
    pin_key_frame_permutation,
    pin_per_head_masks_match_sdpa,
]


# ---- pins of the log-sum-exp output: lse(q, k, mask, T, scale) -> [B, H, S] --------

def pin_lse_dense_matches_logsumexp(lse):
    rng = np.random.default_rng(10)
    B, H, F, T, d = 1, 2, 3, 4, 8
    q, k = (_rand(rng, B, H, F * T, d) for _ in range(2))
    scale = 0.45
    ref = torch.logsumexp(scale * torch.from_numpy(q) @ torch.from_numpy(k).transpose(-1, -2), dim=-1).numpy()
    got = lse(q, k, np.ones((F, F), np.uint8), T, scale)
    assert np.max(np.abs(got - ref)) < TOL


def pin_lse_bruteforce(lse):
    """Pure-Python log(sum(exp)) over the kept keys, -inf for rows keeping nothing,
    with a different mask per head."""
    rng = np.random.default_rng(11)
    H, F, T, d = 2, 3, 2, 3
    masks = np.array([[[1, 0, 1], [0, 0, 0], [1, 1, 0]], [[0, 1, 0], [1, 1, 1], [0, 0, 1]]], np.uint8)
    q, k = (_rand(rng, 1, H, F * T, d) for _ in range(2))
    got = lse(q, k, masks, T, 1.3)
    for h in range(H):
        for s in range(F * T):
            kept = [t for t in range(F * T) if masks[h][s // T][t // T]]
            if not kept:
                assert got[0, h, s] == -np.inf
                continue
            z = sum(math.exp(1.3 * sum(q[0, h, s, c] * k[0, h, t, c] for c in range(d))) for t in kept)
            assert abs(got[0, h, s] - math.log(z)) < TOL, (h, s)


def pin_lse_uniform(lse):
    """Q = 0: every logit is 0, so lse = log(number of kept keys) = log(T * kept frames)."""
    rng = np.random.default_rng(12)
    F, T, d = 5, 7, 4
    mask = (rng.random((F, F)) < 0.5).astype(np.uint8)
    mask[0, :] = 1
    k = _rand(rng, 1, 1, F * T, d)
    got = lse(np.zeros_like(k), k, mask, T, 0.9)
    for i in range(F):
        n = int(mask[i].sum())
        expect = math.log(T * n) if n else -np.inf
        assert np.all(got[0, 0, i * T:(i + 1) * T] == expect) or np.max(np.abs(got[0, 0, i * T:(i + 1) * T] - expect)) < TOL


LSE_PINS = [pin_lse_dense_matches_logsumexp, pin_lse_bruteforce, pin_lse_uniform]


# ---- pins of the gradients: bwd(q, k, v, dout, mask, T, scale) -> (dq, dk, dv) -------

def _autograd_masked(q, k, v, dout, mask, T, scale):
    """torch autograd (float64) through SDPA with the token mask of each head; rows that
    keep nothing contribute nothing."""
    B, H, S, d = q.shape
    F = S // T
    frame = np.arange(S) // T
    grads = [np.zeros_like(q) for _ in range(3)]
    for h in range(H):
        m = np.asarray(mask if np.ndim(mask) == 2 else mask[h], dtype=bool)
        tok = m[frame][:, frame]
        empty = ~tok.any(axis=1)
        tok[empty, :] = True
        qt, kt, vt = (torch.tensor(x[:, h:h + 1], requires_grad=True) for x in (q, k, v))
        out = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=torch.from_numpy(tok), scale=scale)
        g = torch.from_numpy(dout[:, h:h + 1].copy())
        g[:, :, torch.from_numpy(empty)] = 0.0
        out.backward(g)
        for dst, t in zip(grads, (qt, kt, vt)):
            dst[:, h:h + 1] = t.grad.numpy()
    return grads


def pin_bwd_matches_autograd(bwd):
    rng = np.random.default_rng(20)
    for (B, H, F, T, d, p) in [(1, 2, 3, 4, 8, 1.0), (2, 2, 4, 3, 4, 0.5), (1, 3, 5, 2, 6, 0.3)]:
        q, k, v, g = (_rand(rng, B, H, F * T, d) for _ in range(4))
        masks = (rng.random((H, F, F)) < p).astype(np.uint8)
        masks[0, 0, :] = 0
        got = bwd(q, k, v, g, masks, T, 0.55)
        ref = _autograd_masked(q, k, v, g, masks, T, 0.55)
        for a, r, name in zip(got, ref, "qkv"):
            assert np.max(np.abs(a - r)) < 1e-11, f"d{name}"


def pin_bwd_bruteforce(bwd):
    """Pure-Python chain rule through the softmax, token by token."""
    rng = np.random.default_rng(21)
    F, T, d, scale = 3, 2, 3, 0.8
    mask = np.array([[1, 0, 1], [0, 0, 0], [1, 1, 0]], np.uint8)
    q, k, v, g = (_rand(rng, 1, 1, F * T, d, 0.7) for _ in range(4))
    dq, dk, dv = bwd(q, k, v, g, mask, T, scale)
    S = F * T
    edq, edk, edv = np.zeros((S, d)), np.zeros((S, d)), np.zeros((S, d))
    for s in range(S):
        kept = [t for t in range(S) if mask[s // T][t // T]]
        if not kept:
            continue
        w = {t: math.exp(scale * sum(q[0, 0, s, c] * k[0, 0, t, c] for c in range(d))) for t in kept}
        z = sum(w.values())
        p = {t: w[t] / z for t in kept}
        out = [sum(p[t] * v[0, 0, t, c] for t in kept) for c in range(d)]
        dp = {t: sum(g[0, 0, s, c] * v[0, 0, t, c] for c in range(d)) for t in kept}
        big_d = sum(g[0, 0, s, c] * out[c] for c in range(d))
        for t in kept:
            ds = p[t] * (dp[t] - big_d)
            for c in range(d):
                edq[s, c] += scale * ds * k[0, 0, t, c]
                edk[t, c] += scale * ds * q[0, 0, s, c]
                edv[t, c] += p[t] * g[0, 0, s, c]
    for a, e in ((dq, edq), (dk, edk), (dv, edv)):
        assert np.max(np.abs(a[0, 0] - e)) < TOL


def pin_bwd_uniform_weights(bwd):
    """Q = 0: P is uniform over the kept keys, so dv_t = sum over the rows keeping t of
    dO_s / n_s (n_s = kept keys of s) and dk = 0 (all scores equal, dS sums to zero
    against equal q = 0)."""
    rng = np.random.default_rng(22)
    F, T, d = 4, 3, 5
    mask = (rng.random((F, F)) < 0.5).astype(np.uint8)
    mask[0, :] = 1
    k, v, g = (_rand(rng, 1, 1, F * T, d) for _ in range(3))
    dq, dk, dv = bwd(np.zeros_like(k), k, v, g, mask, T, 0.9)
    assert np.max(np.abs(dk)) < TOL
    expect = np.zeros((F * T, d))
    for s in range(F * T):
        kept = [t for t in range(F * T) if mask[s // T][t // T]]
        for t in kept:
            expect[t] += g[0, 0, s] / len(kept)
    assert np.max(np.abs(dv[0, 0] - expect)) < TOL


BWD_PINS = [pin_bwd_matches_autograd, pin_bwd_bruteforce, pin_bwd_uniform_weights]


# ---- pins of the MM-DiT form: fn(q, k, v, mask, T, P, scale) -> out --------------------

def _mmdit_token_mask(mask_h, F, T, P):
    """Boolean [S, S] token mask: text rows and text columns all kept, video-video part
    from the frame mask."""
    S = P + F * T
    tok = np.zeros((S, S), dtype=bool)
    tok[:P, :] = True
    tok[:, :P] = True
    fr = np.arange(F * T) // T
    tok[P:, P:] = np.asarray(mask_h, dtype=bool)[fr][:, fr]
    return tok


def pin_mmdit_matches_sdpa_token_mask(fn):
    rng = np.random.default_rng(30)
    for (B, H, F, T, P, d) in [(1, 2, 3, 4, 5, 8), (2, 3, 4, 3, 1, 6), (1, 2, 5, 2, 7, 4)]:
        q, k, v = (_rand(rng, B, H, P + F * T, d) for _ in range(3))
        masks = (rng.random((H, F, F)) < 0.4).astype(np.uint8)
        masks[0, 1, :] = 0  # a video frame keeping no video frame still sees the text
        got = fn(q, k, v, masks, T, P, 0.7)
        for h in range(H):
            tok = torch.from_numpy(_mmdit_token_mask(masks[h], F, T, P))
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q[:, h]), torch.from_numpy(k[:, h]), torch.from_numpy(v[:, h]),
                attn_mask=tok, scale=0.7).numpy()
            assert np.max(np.abs(got[:, h] - ref)) < TOL


def pin_mmdit_dense_is_plain_attention_over_all_tokens(fn):
    rng = np.random.default_rng(31)
    B, H, F, T, P, d = 2, 2, 3, 5, 4, 8
    q, k, v = (_rand(rng, B, H, P + F * T, d) for _ in range(3))
    got = fn(q, k, v, np.ones((F, F), np.uint8), T, P, 0.3)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), scale=0.3).numpy()
    assert np.max(np.abs(got - ref)) < TOL


def pin_mmdit_bruteforce(fn):
    """Token by token in pure Python, from the stated rule."""
    rng = np.random.default_rng(32)
    F, T, P, d, scale = 3, 2, 2, 3, 0.9
    mask = np.array([[1, 0, 0], [0, 0, 0], [1, 1, 0]], np.uint8)
    q, k, v = (_rand(rng, 1, 1, P + F * T, d, 0.8) for _ in range(3))
    got = fn(q, k, v, mask, T, P, scale)
    S = P + F * T
    for s in range(S):
        if s < P:
            keys = list(range(S))
        else:
            i = (s - P) // T
            keys = [t for t in range(S) if t < P or mask[i][(t - P) // T]]
        w = [math.exp(scale * sum(q[0, 0, s, c] * k[0, 0, t, c] for c in range(d))) for t in keys]
        z = sum(w)
        for c in range(d):
            ref = sum(wi * v[0, 0, t, c] for wi, t in zip(w, keys)) / z
            assert abs(got[0, 0, s, c] - ref) < TOL


def pin_mmdit_text_queries_ignore_the_mask(fn):
    """Invariant: text rows attend to everything, so no mask changes them; and with
    identical video frames a video row's output depends only on how many frames it
    keeps (here: frame 1 keeps one frame, frame 2 keeps one other frame)."""
    rng = np.random.default_rng(33)
    F, T, P, d = 3, 4, 3, 5
    q, k, v = (_rand(rng, 1, 1, P + F * T, d) for _ in range(3))
    a = fn(q, k, v, np.eye(F, dtype=np.uint8), T, P, 0.5)
    b = fn(q, k, v, np.ones((F, F), np.uint8), T, P, 0.5)
    assert np.max(np.abs(a[0, 0, :P] - b[0, 0, :P])) < TOL
    kk, vv = k.copy(), v.copy()
    for j in range(1, F):
        kk[0, 0, P + j * T:P + (j + 1) * T] = kk[0, 0, P:P + T]
        vv[0, 0, P + j * T:P + (j + 1) * T] = vv[0, 0, P:P + T]
    m = np.array([[1, 0, 0], [0, 0, 1], [1, 0, 0]], np.uint8)
    got = fn(q, kk, vv, m, T, P, 0.5)
    m2 = np.array([[1, 0, 0], [1, 0, 0], [0, 1, 0]], np.uint8)
    got2 = fn(q, kk, vv, m2, T, P, 0.5)
    assert np.max(np.abs(got[0, 0, P + T:] - got2[0, 0, P + T:])) < TOL


MMDIT_PINS = [pin_mmdit_matches_sdpa_token_mask, pin_mmdit_dense_is_plain_attention_over_all_tokens,
              pin_mmdit_bruteforce, pin_mmdit_text_queries_ignore_the_mask]


def pin_mmdit_lse(lse_fn):
    """The MM-DiT log-sum-exp against torch.logsumexp over the token mask."""
    rng = np.random.default_rng(34)
    B, H, F, T, P, d = 1, 2, 4, 3, 5, 6
    q, k = (_rand(rng, B, H, P + F * T, d) for _ in range(2))
    masks = (rng.random((H, F, F)) < 0.5).astype(np.uint8)
    got = lse_fn(q, k, masks, T, P, 0.8)
    for h in range(H):
        tok = torch.from_numpy(_mmdit_token_mask(masks[h], F, T, P))
        logits = 0.8 * torch.from_numpy(q[:, h]) @ torch.from_numpy(k[:, h]).transpose(-1, -2)
        ref = torch.logsumexp(logits.masked_fill(~tok, float("-inf")), dim=-1).numpy()
        assert np.max(np.abs(got[:, h] - ref)) < TOL


def pin_mmdit_bwd_matches_autograd(bwd):
    """fn(q, k, v, dout, mask, T, P, scale) -> (dq, dk, dv) against torch autograd through
    SDPA with the MM-DiT token mask (float64), per-head masks."""
    rng = np.random.default_rng(40)
    for (B, H, F, T, P, d) in [(1, 2, 3, 4, 5, 8), (2, 2, 4, 3, 1, 4), (1, 3, 3, 2, 6, 6)]:
        q, k, v, g = (_rand(rng, B, H, P + F * T, d) for _ in range(4))
        masks = (rng.random((H, F, F)) < 0.4).astype(np.uint8)
        masks[0, 1, :] = 0
        got = bwd(q, k, v, g, masks, T, P, 0.6)
        for h in range(H):
            tok = torch.from_numpy(_mmdit_token_mask(masks[h], F, T, P))
            qt, kt, vt = (torch.tensor(x[:, h], requires_grad=True) for x in (q, k, v))
            out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=tok, scale=0.6)
            out.backward(torch.from_numpy(g[:, h].copy()))
            for a, t in zip(got, (qt, kt, vt)):
                assert np.max(np.abs(a[:, h] - t.grad.numpy())) < 1e-11


def pin_mmdit_bwd_bruteforce(bwd):
    rng = np.random.default_rng(41)
    F, T, P, d, scale = 2, 2, 2, 3, 0.7
    mask = np.array([[0, 1], [0, 0]], np.uint8)
    q, k, v, g = (_rand(rng, 1, 1, P + F * T, d, 0.8) for _ in range(4))
    dq, dk, dv = bwd(q, k, v, g, mask, T, P, scale)
    S = P + F * T
    edq, edk, edv = np.zeros((S, d)), np.zeros((S, d)), np.zeros((S, d))
    for s in range(S):
        keys = list(range(S)) if s < P else [t for t in range(S) if t < P or mask[(s - P) // T][(t - P) // T]]
        w = {t: math.exp(scale * sum(q[0, 0, s, c] * k[0, 0, t, c] for c in range(d))) for t in keys}
        z = sum(w.values())
        p = {t: w[t] / z for t in keys}
        out = [sum(p[t] * v[0, 0, t, c] for t in keys) for c in range(d)]
        dp = {t: sum(g[0, 0, s, c] * v[0, 0, t, c] for c in range(d)) for t in keys}
        delta = sum(g[0, 0, s, c] * out[c] for c in range(d))
        for t in keys:
            ds = p[t] * (dp[t] - delta)
            for c in range(d):
                edq[s, c] += scale * ds * k[0, 0, t, c]
                edk[t, c] += scale * ds * q[0, 0, s, c]
                edv[t, c] += p[t] * g[0, 0, s, c]
    for a, e in ((dq, edq), (dk, edk), (dv, edv)):
        assert np.max(np.abs(a[0, 0] - e)) < TOL


MMDIT_BWD_PINS = [pin_mmdit_bwd_matches_autograd, pin_mmdit_bwd_bruteforce]
