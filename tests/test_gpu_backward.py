"""Parity of the gfx950 gradient kernels (tile_attn_bwd) with the float64 oracle.

The GPU forward (tile_attn_fwd_heads) supplies out and the row log-sum-exp, as a
training step would; the oracle recomputes everything in float64 from the same
bf16 q, k, v and dout. Small problems are compared in full, the measured shapes
on sampled query and key rows.
"""
import numpy as np
import pytest

import workloads
from oracle import backward as ob
from oracle import masks as om
from oracle import mmdit as ommd
from tests.gpu_helpers import from_dev, to_dev, widen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402

# Gate for bf16 gradients. P and dS enter the matrix cores as bf16 (relative
# rounding 2^-9 each), delta is formed from the bf16 forward output, and the
# results are rounded to bf16 (2^-9 of each value): an honest path sits near 3e-3
# relative RMS. Errors are measured against the tensor's own scale, since gradient
# magnitudes vary with the number of queries that keep a key.
GRAD_REL_RMS = 1e-2
GRAD_MAX_REL = 2e-2  # max abs error / max abs reference


def grad_errors(got_bits, ref):
    got = widen(got_bits)
    diff = np.abs(got - ref)
    peak = float(np.max(np.abs(ref))) if ref.size else 0.0
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    return {
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "max_rel": float(diff.max()) / peak if peak > 0 else float(diff.max() if diff.size else 0.0),
        "rel_rms": float(np.sqrt(np.mean(diff * diff))) / rms if rms > 0 else 0.0,
        "peak": peak,
        "finite": bool(np.all(np.isfinite(got))),
    }


def assert_grad(got_bits, ref, what):
    e = grad_errors(got_bits, ref)
    print(f"[grad] {what} {e}", flush=True)
    assert e["finite"], f"{what}: non-finite gradient"
    if e["peak"] == 0.0:
        assert e["max_abs"] == 0.0, f"{what}: expected exact zeros"
        return e
    assert e["max_rel"] <= GRAD_MAX_REL, f"{what}: max abs / peak {e['max_rel']}"
    assert e["rel_rms"] <= GRAD_REL_RMS, f"{what}: rel rms {e['rel_rms']}"
    return e


def make_grad(B, H, S, d, seed):
    rng = np.random.default_rng(seed)
    return workloads.f32_to_bf16_bits(rng.standard_normal((B, H, S, d)).astype(np.float32))


def run_gpu_bwd(qb, kb, vb, gb, masks, T, scale, stream=None):
    B, H, S, d = qb.shape
    F = S // T
    q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
    s = stream or torch.cuda.current_stream()
    out = torch.empty_like(q)
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    grads = [torch.full_like(q, float("nan")) for _ in range(3)]
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, masks, scale, lse, s)
        ta.tile_attn_bwd(q, k, v, out, g, lse, *grads, B, H, F, T, d, masks, scale, s)
    torch.cuda.synchronize()
    return tuple(from_dev(x) for x in grads)


def full_check(qb, kb, vb, gb, masks, T, scale, what):
    print(f"[case] {what} shape={qb.shape} T={T}", flush=True)
    got = run_gpu_bwd(qb, kb, vb, gb, masks, T, scale)
    ref = ob.attention_backward(qb, kb, vb, gb, masks, T, scale)
    for name, a, r in zip(("dq", "dk", "dv"), got, ref):
        assert_grad(a, r, f"{what}-{name}")
    return got


def _masks(F, H, seed):
    rng = np.random.default_rng(seed)
    ms = (rng.random((H, F, F)) < 0.45).astype(np.uint8)
    ms[0, 1, :] = 0  # a query frame that keeps nothing
    ms[-1, :, 2] = 0  # a key frame nobody keeps
    return ms


@pytest.mark.parametrize("d", [64, 96, 128])
def test_bwd_random_per_head_masks(d):
    B, H, F, T = 2, 3, 5, 130
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=60 + d, dist="frame_shift")
    gb = make_grad(B, H, F * T, d, 61 + d)
    full_check(qb, kb, vb, gb, _masks(F, H, d), T, d ** -0.5, f"bwd-heads-d{d}")


@pytest.mark.parametrize("d", [64, 96, 128])
@pytest.mark.parametrize("T", [1, 17, 63, 64, 65, 129, 200, 257])
def test_bwd_ragged_tails(d, T):
    B, H, F = 1, 2, 3
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T * 3 + d)
    gb = make_grad(B, H, F * T, d, T + d)
    mask = np.array([[1, 0, 1], [1, 1, 0], [0, 1, 1]], np.uint8)
    full_check(qb, kb, vb, gb, mask, T, d ** -0.5, f"bwd-tails-d{d}-T{T}")


@pytest.mark.parametrize("form", ["col", "sym"])
@pytest.mark.parametrize("d", [64, 96, 128])
def test_bwd_split_frames(form, d):
    """Heavy rows (sym) and heavy columns (both forms: every query frame keeps frame 0)
    are split into pieces whose fp32 partials are summed."""
    B, H, F, T = 2, 2, 10, 150
    mask = om.tile_mask(F, 1, form)
    assert ta.tile_attn_plan(mask.T.copy())[1] > 0
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=70 + d)
    gb = make_grad(B, H, F * T, d, 71 + d)
    full_check(qb, kb, vb, gb, mask, T, d ** -0.5, f"bwd-split-{form}-d{d}")


@pytest.mark.parametrize("scale", [-0.1, 0.0, 0.35])
def test_bwd_scales(scale):
    B, H, F, T, d = 1, 2, 5, 70, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=80)
    gb = make_grad(B, H, F * T, d, 81)
    masks = np.stack([om.tile_mask(F, 1, "sym"), om.tile_mask(F, 2, "col")])
    got = full_check(qb, kb, vb, gb, masks, T, scale, f"bwd-scale{scale}")
    if scale == 0.0:
        assert not np.any(widen(got[0])) and not np.any(widen(got[1]))


def test_bwd_unkept_frames_get_exact_zeros():
    B, H, F, T, d = 1, 2, 4, 100, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=90)
    gb = make_grad(B, H, F * T, d, 91)
    mask = om.tile_mask(F, 1, "col")
    mask[2, :] = 0  # query frame 2 keeps nothing
    mask[:, 3] = 0  # nobody keeps key frame 3
    dq, dk, dv = run_gpu_bwd(qb, kb, vb, gb, mask, T, d ** -0.5)
    assert np.all(widen(dq[:, :, 2 * T:3 * T]) == 0)
    assert np.all(widen(dk[:, :, 3 * T:]) == 0) and np.all(widen(dv[:, :, 3 * T:]) == 0)


def test_bwd_skipped_tiles_are_never_read():
    """NaN-poison the k, v of a frame (key side) or the q, dout of a frame (query
    side) for the gradient pass only: every gradient that does not depend on the
    poisoned tiles must stay bit-identical, so they are skipped, not masked."""
    B, H, F, T, d = 1, 2, 6, 200, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=92)
    gb = make_grad(B, H, F * T, d, 93)
    mask = om.tile_mask(F, 2, "col")  # G = {0, 3}
    scale = d ** -0.5
    q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
    out = torch.empty_like(q)
    lse = torch.empty((B, H, F * T), dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, mask, scale, lse, None)

    def grads(qq, kk, vv, gg):
        res = [torch.empty_like(q) for _ in range(3)]
        ta.tile_attn_bwd(qq, kk, vv, out, gg, lse, *res, B, H, F, T, d, mask, scale, None)
        torch.cuda.synchronize()
        return [from_dev(x) for x in res]

    base = grads(q, k, v, g)
    nan = 0x7FC0
    # key side: poison k, v of frame 4 (kept only by query frame 4)
    kp, vp = kb.copy(), vb.copy()
    kp[:, :, 4 * T:5 * T] = nan
    vp[:, :, 4 * T:5 * T] = nan
    got = grads(q, to_dev(kp), to_dev(vp), g)
    for i in range(F):
        if not mask[i, 4]:
            assert np.array_equal(got[0][:, :, i * T:(i + 1) * T], base[0][:, :, i * T:(i + 1) * T]), i
    for j in range(F):
        if j != 4:
            for t in (1, 2):
                assert np.array_equal(got[t][:, :, j * T:(j + 1) * T], base[t][:, :, j * T:(j + 1) * T]), j
    # query side: poison q, dout of frame 5 (keeps frames 0, 3, 5)
    qp, gp = qb.copy(), gb.copy()
    qp[:, :, 5 * T:6 * T] = nan
    gp[:, :, 5 * T:6 * T] = nan
    got = grads(to_dev(qp), k, v, to_dev(gp))
    for j in range(F):
        if not mask[5, j]:
            for t in (1, 2):
                assert np.array_equal(got[t][:, :, j * T:(j + 1) * T], base[t][:, :, j * T:(j + 1) * T]), j
    for i in range(5):
        assert np.array_equal(got[0][:, :, i * T:(i + 1) * T], base[0][:, :, i * T:(i + 1) * T]), i


def test_bwd_repeat_calls_bitwise_equal_and_side_stream():
    B, H, F, T, d = 1, 3, 8, 300, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=94)
    gb = make_grad(B, H, F * T, d, 95)
    mask = om.tile_mask(F, 1, "sym")
    a = run_gpu_bwd(qb, kb, vb, gb, mask, T, d ** -0.5)
    b = run_gpu_bwd(qb, kb, vb, gb, mask, T, d ** -0.5, stream=torch.cuda.Stream())
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_bwd_last_key_block_full_frames():
    """T = 3600: the last key workgroup of each frame holds 16 keys and the last
    query tile 16 queries; every gradient row of two heads is compared."""
    B, H, F, T, d = 1, 2, 3, 3600, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=96)
    gb = make_grad(B, H, F * T, d, 97)
    full_check(qb, kb, vb, gb, om.tile_mask(F, 1, "col"), T, d ** -0.5, "bwd-3600")


# Every workload the benchmark times for the gradients: the 93-frame and 29-frame shapes,
# the frame-correlated sweep data, one GPU's head share, the 48-frame long horizon (T =
# 1200, two global frames) and 128-wide heads (split dV and dK key-side passes).
FULL_CASES = [("93f", "col", 1), ("93f", "sym", 1), ("29f", "col", 1), ("sweep", "sym", 2),
              ("sp_share", "sym", 1), ("long", "col", 2), ("93f_d128", "col", 1)]


@pytest.mark.parametrize("name,form,g", FULL_CASES, ids=[f"{a}-{b}-g{c}" for a, b, c in FULL_CASES])
def test_bwd_full_size_sampled(name, form, g):
    """The measured shapes in the benchmark's launch configuration: dq on sampled
    query rows and dk, dv on sampled key rows (the heavy global frame 0, an ordinary
    frame and the last frame, including each frame's ragged last rows) of two heads."""
    w = workloads.WORKLOADS[name]
    print(f"[case] bwd full {name} {form} g={g}", flush=True)
    qb, kb, vb = workloads.make_workload_qkv(w)
    gb = make_grad(w.B, w.H, w.F * w.T, w.d, 98)
    mask = om.tile_mask(w.F, g, form)
    dq, dk, dv = run_gpu_bwd(qb, kb, vb, gb, mask, w.T, w.scale())
    rng = np.random.default_rng(99)
    heads = [0, w.H - 1]
    rows_q, rows_k = [], []
    for h in heads:
        for f in range(w.F):
            for r in {0, w.T - 1, int(rng.integers(0, w.T))}:
                rows_q.append((0, h, f * w.T + r))
        for f in (0, 1, w.F - 1):
            for r in {0, 255, 256, w.T - 17, w.T - 1, int(rng.integers(0, w.T))}:
                rows_k.append((0, h, f * w.T + r))
    bq, hq, sq = (np.array(x) for x in zip(*rows_q))
    bk, hk, sk = (np.array(x) for x in zip(*rows_k))
    rq, rk, rv = ob.attention_backward_rows(qb, kb, vb, gb, mask, w.T, w.scale(), bq, hq, sq, bk, hk, sk)
    assert_grad(dq[bq, hq, sq], rq, f"{name}-{form}-dq")
    assert_grad(dk[bk, hk, sk], rk, f"{name}-{form}-dk")
    assert_grad(dv[bk, hk, sk], rv, f"{name}-{form}-dv")
    for x in (dq, dk, dv):
        assert np.all(np.isfinite(widen(x[:, :, :: max(1, w.T // 7)])))


# ---- the MM-DiT form (text prefix) ------------------------------------------------------

def run_gpu_bwd_mmdit(qb, kb, vb, gb, masks, T, P, scale):
    B, H, S, d = qb.shape
    F = (S - P) // T
    q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
    out = torch.empty_like(q)
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    grads = [torch.full_like(q, float("nan")) for _ in range(3)]
    s = torch.cuda.current_stream()
    ta.tile_attn_fwd_mmdit(q, k, v, out, B, H, F, T, P, d, masks, scale, lse, s)
    ta.tile_attn_bwd_mmdit(q, k, v, out, g, lse, *grads, B, H, F, T, P, d, masks, scale, s)
    torch.cuda.synchronize()
    return tuple(from_dev(x) for x in grads)


@pytest.mark.parametrize("d", [64, 96, 128])
@pytest.mark.parametrize("T,P", [(130, 17), (64, 226), (65, 1), (40, 300)])
def test_bwd_mmdit_small(d, T, P):
    B, H, F = 2, 2, 4
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T + P + d, prefix=P)
    gb = make_grad(B, H, P + F * T, d, T * P + d)
    masks = _masks(F, H, T + P)
    print(f"[case] bwd mmdit d={d} T={T} P={P}", flush=True)
    got = run_gpu_bwd_mmdit(qb, kb, vb, gb, masks, T, P, d ** -0.5)
    ref = ommd.attention_backward_mmdit(qb, kb, vb, gb, masks, T, P, d ** -0.5)
    for name, a, r in zip(("dq", "dk", "dv"), got, ref):
        assert_grad(a, r, f"bwd-mmdit-d{d}-T{T}-P{P}-{name}")


def test_bwd_mmdit_without_text_matches_plain_bitwise():
    B, H, F, T, d = 1, 2, 5, 150, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=101)
    gb = make_grad(B, H, F * T, d, 102)
    mask = om.tile_mask(F, 1, "sym")
    a = run_gpu_bwd_mmdit(qb, kb, vb, gb, mask, T, 0, d ** -0.5)
    b = run_gpu_bwd(qb, kb, vb, gb, mask, T, d ** -0.5)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("k", [1, 12])
def test_bwd_mmdit_cog_shape_sampled(k):
    """CogVideoX-5B shape (226 text tokens, 13 x 1350 video tokens, 48 heads of 64),
    sym masks: text and video query rows and key rows (text keys are kept by every
    query) of two heads."""
    w = workloads.WORKLOADS["cog"]
    qb, kb, vb = workloads.make_workload_qkv(w)
    gb = make_grad(w.B, w.H, w.S, w.d, 103)
    mask = om.tile_mask(w.F, k, "sym")
    print(f"[case] bwd cog k={k}", flush=True)
    dq, dk, dv = run_gpu_bwd_mmdit(qb, kb, vb, gb, mask, w.T, w.prefix, w.scale())
    rng = np.random.default_rng(k)
    rows = []
    for h in (0, w.H - 1):
        for s in list(range(0, w.prefix, 37)) + [w.prefix - 1]:
            rows.append((0, h, s))
        for f in (0, 1, w.F - 1):
            for r in {0, w.T - 1, int(rng.integers(0, w.T))}:
                rows.append((0, h, w.prefix + f * w.T + r))
    b, h, s = (np.array(x) for x in zip(*rows))
    rq, rk, rv = ommd.attention_backward_mmdit_rows(qb, kb, vb, gb, mask, w.T, w.prefix, w.scale(),
                                                    b, h, s, b, h, s)
    assert_grad(dq[b, h, s], rq, f"cog-k{k}-dq")
    assert_grad(dk[b, h, s], rk, f"cog-k{k}-dk")
    assert_grad(dv[b, h, s], rv, f"cog-k{k}-dv")


def test_all_zero_mask_forward_and_gradients():
    """A mask that keeps nothing: zero output, -inf log-sum-exp, zero gradients (every
    output written over a NaN fill)."""
    B, H, F, T, d = 1, 2, 3, 100, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=110)
    gb = make_grad(B, H, F * T, d, 111)
    mask = np.zeros((F, F), np.uint8)
    q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
    out = torch.full_like(q, float("nan"))
    lse = torch.zeros((B, H, F * T), dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, mask, 0.125, lse, None)
    grads = [torch.full_like(q, float("nan")) for _ in range(3)]
    ta.tile_attn_bwd(q, k, v, out, g, lse, *grads, B, H, F, T, d, mask, 0.125, None)
    torch.cuda.synchronize()
    assert not np.any(widen(from_dev(out)))
    assert np.all(np.isneginf(lse.cpu().numpy()))
    for x in grads:
        assert not np.any(widen(from_dev(x)))


def test_calls_of_growing_size_share_one_stream_without_waits():
    """Forward and gradient calls of increasing workspace needs queued back to back on
    one stream (each grows the workspace; the old ones stay alive): every result
    matches the oracle."""
    d, scale = 64, 0.125
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    cases = [(1, 2, 6, 90, "sym"), (2, 2, 8, 150, "col"), (1, 3, 10, 200, "sym")]
    results = []
    with torch.cuda.stream(s):
        for (B, H, F, T, form) in cases:
            qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=F * T)
            gb = make_grad(B, H, F * T, d, F + T)
            mask = om.tile_mask(F, 1, form)
            q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
            out = torch.empty_like(q)
            lse = torch.empty((B, H, F * T), dtype=torch.float32, device="cuda")
            grads = [torch.empty_like(q) for _ in range(3)]
            ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, mask, scale, lse, s)
            ta.tile_attn_bwd(q, k, v, out, g, lse, *grads, B, H, F, T, d, mask, scale, s)
            results.append((qb, kb, vb, gb, mask, T, out, grads))
    torch.cuda.synchronize()
    for qb, kb, vb, gb, mask, T, out, grads in results:
        from oracle import attention as oa
        from tests.gpu_helpers import assert_parity
        assert_parity(from_dev(out), oa.attention(qb, kb, vb, mask, T, scale), "stream-fwd")
        ref = ob.attention_backward(qb, kb, vb, gb, mask, T, scale)
        for name, a, r in zip(("dq", "dk", "dv"), grads, ref):
            assert_grad(from_dev(a), r, f"stream-{name}")
