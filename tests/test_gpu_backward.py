"""Parity of the gfx950 gradient kernels (tile_attn_bwd) with the float64 oracle.

The GPU forward (tile_attn_fwd_heads) supplies out and the row log-sum-exp, as a
training step would; the oracle recomputes everything in float64 from the same
bf16 q, k, v and dout. Small problems are compared in full, the measured shapes
on sampled query and key rows.
"""
import numpy as np
import pytest

import workloads
from oracle import attention as oa
from oracle import backward as ob
from oracle import masks as om
from oracle import mmdit as ommd
from tests.gpu_helpers import from_dev, to_dev, upstream_grad, widen, workload_inputs

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
        "mean_abs": float(diff.mean()) if diff.size else 0.0,
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


# Every (workload, mask form, g) the benchmark times for the gradients (bench.py
# ALL_CASES with --pass bwd), with the dense control of each workload: the 93-frame and
# 29-frame shapes, the frame-correlated sweep data, one GPU's head share, the 48-frame
# long horizon (T = 1200, two global frames) and 128-wide heads (split dV and dK
# key-side passes). Rows of the masks with many kept pairs per key check dk and dv on
# one head, to keep the float64 oracle's work per case near the others'.
FULL_CASES = [
    ("29f", "col", 1), ("29f", "sym", 1), ("29f", "dense", 0),
    ("93f", "col", 1), ("93f", "sym", 1), ("93f", "dense", 0),
    ("sweep", "col", 1), ("sweep", "col", 2), ("sweep", "col", 4), ("sweep", "col", 8),
    ("sweep", "sym", 2), ("sweep", "sym", 4), ("sweep", "sym", 8), ("sweep", "dense", 0),
    ("sp_share", "col", 1), ("sp_share", "sym", 1), ("sp_share", "dense", 0),
    ("long", "col", 2), ("long", "sym", 2), ("long", "dense", 0),
    ("93f_d128", "col", 1), ("93f_d128", "sym", 1), ("93f_d128", "dense", 0),
]


def _bwd_full(name, form, g):
    w = workloads.WORKLOADS[name]
    qb, kb, vb = workload_inputs(name)
    gb = upstream_grad(qb.shape, 98)
    mask = np.ones((w.F, w.F), np.uint8) if form == "dense" else om.tile_mask(w.F, g, form)
    return w, qb, kb, vb, gb, mask, run_gpu_bwd(qb, kb, vb, gb, mask, w.T, w.scale())


@pytest.mark.parametrize("name,form,g", [c for c in FULL_CASES if c[1] != "dense" or c[0] == "29f"],
                         ids=[f"{a}-{b}-g{c}" for a, b, c in FULL_CASES if b != "dense" or a == "29f"])
def test_bwd_full_size_sampled(name, form, g):
    """The measured shapes in the benchmark's launch configuration: dq on sampled
    query rows and dk, dv on sampled key rows (the heavy global frame 0, an ordinary
    frame and the last frame, including each frame's ragged last rows)."""
    print(f"[case] bwd full {name} {form} g={g}", flush=True)
    w, qb, kb, vb, gb, mask, (dq, dk, dv) = _bwd_full(name, form, g)
    rng = np.random.default_rng(99)
    heads = [0, w.H - 1]
    # a key row's gradient sums over every query frame that keeps its frame
    key_heads = heads if np.count_nonzero(mask) <= 2 * 70 else heads[:1]
    rows_q, rows_k = [], []
    for h in heads:
        for f in range(w.F):
            for r in {0, w.T - 1, int(rng.integers(0, w.T))}:
                rows_q.append((0, h, f * w.T + r))
    for h in key_heads:
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


@pytest.mark.parametrize("name", [c[0] for c in FULL_CASES if c[1] == "dense" and c[0] != "29f"])
def test_bwd_dense_full_size(name):
    """The dense control's gradients at the full shapes (the 29-frame one is checked row
    by row above). dq on sampled query rows of two heads against the oracle; a key row's
    oracle gradient would need the whole attention of its head (about 3e12 float64
    FLOP at 93 frames), so dk and dv are checked, over every head, by two identities
    that hold for any mask at any size:
      - the scores' gradients of one query sum to zero over its kept keys
        (sum_t dS_st = D_s - D_s), so the keys' dk sum to zero;
      - the attention weights of one query sum to one, so the keys' dv sum to the sum
        of dO over the queries.
    In bf16 the first sum moves off zero mainly through delta, which is formed from
    the bf16 forward output: D_s errs by about 2^-8 |O_s| |dO_s| / sqrt(3), and these
    errors enter sum_t dk_t weighted by scale * q_s with random signs. The bound takes
    |O_s| from the oracle's rows, plus the bf16 rounding of the S summed rows. Dropping
    delta altogether moves the sum by |D_s| itself, about 90 times further."""
    print(f"[case] bwd dense full {name}", flush=True)
    w, qb, kb, vb, gb, mask, (dq, dk, dv) = _bwd_full(name, "dense", 0)
    rng = np.random.default_rng(100)
    rows_q = [(0, h, f * w.T + r) for h in (0, w.H - 1) for f in range(w.F)
              for r in {0, w.T - 1, int(rng.integers(0, w.T))}]
    bq, hq, sq = (np.array(x) for x in zip(*rows_q))
    empty = np.zeros(0, np.int64)
    rq, _, _ = ob.attention_backward_rows(qb, kb, vb, gb, mask, w.T, w.scale(), bq, hq, sq,
                                          empty, empty, empty)
    assert_grad(dq[bq, hq, sq], rq, f"{name}-dense-dq")
    o_rows = oa.attention_rows(qb, kb, vb, mask, w.T, w.scale(), bq, hq, sq)
    o_norm = float(np.sqrt(np.mean(np.sum(o_rows ** 2, axis=1))))
    worst_k = worst_v = 0.0
    for b in range(w.B):
        for h in range(w.H):
            dk64, dv64, g64, q64 = (widen(x[b, h]) for x in (dk, dv, gb, qb))
            do_norm = float(np.sqrt(np.mean(np.sum(g64 ** 2, axis=1))))
            rms_dk = float(np.sqrt(np.mean(dk64 ** 2)))
            rms_dv = float(np.sqrt(np.mean(dv64 ** 2)))
            rounding = np.sqrt(w.S) * 2.0 ** -9
            tol_k = 6 * (w.scale() * 2.0 ** -8 * o_norm * do_norm / np.sqrt(3)
                         * np.sqrt(np.sum(q64 ** 2, axis=0)) + rounding * rms_dk)
            tol_v = 8 * 2 * rounding * rms_dv + 1e-3
            err_k = np.abs(dk64.sum(axis=0))
            err_v = np.abs(dv64.sum(axis=0) - g64.sum(axis=0))
            worst_k = max(worst_k, float(np.max(err_k / tol_k)))
            worst_v = max(worst_v, float(np.max(err_v / tol_v)))
    print(f"[grad] {name}-dense sums over keys: |sum dk| / bound {worst_k:.3f}, "
          f"|sum dv - sum dO| / bound {worst_v:.3f} (|O| {o_norm:.3e})", flush=True)
    assert worst_k <= 1.0 and worst_v <= 1.0


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


@pytest.mark.parametrize("k", [1, 2, 3, 4, 6, 12, 0])
def test_bwd_mmdit_cog_shape_sampled(k):
    """CogVideoX-5B shape (226 text tokens, 13 x 1350 video tokens, 48 heads of 64),
    sym masks with k global frames (every mask the benchmark times; k = 0 is the dense
    control): text and video query rows and key rows (text keys are kept by every
    query) of two heads."""
    w = workloads.WORKLOADS["cog"]
    qb, kb, vb = workload_inputs("cog")
    gb = upstream_grad(qb.shape, 103)
    mask = om.tile_mask(w.F, k, "sym") if k else np.ones((w.F, w.F), np.uint8)
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
