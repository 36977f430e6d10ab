"""Parity of the gfx950 HIP path with the float64 oracle (needs an MI355X).

Every call goes through the C ABI (via the ctypes binding). Small problems are
compared element by element against the full oracle; the measured workloads are
run at full size in the benchmark's launch configuration and compared on
sampled rows that the oracle computes one by one.
"""
import numpy as np
import pytest

import workloads
from oracle import attention as oa
from oracle import masks as om
from tests.gpu_helpers import (assert_parity, errors, from_dev, sample_rows, to_dev,
                               workload_inputs)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402


def run_gpu(qb, kb, vb, mask, T, scale, dense=False):
    B, H, S, d = qb.shape
    F = S // T
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    if dense:
        ta.dense_attn_fwd(q, k, v, out, B, H, F, T, d, scale, stream)
    else:
        ta.tile_attn_fwd(q, k, v, out, B, H, F, T, d, mask, scale, stream)
    torch.cuda.synchronize()
    return from_dev(out)


def full_check(qb, kb, vb, mask, T, scale, what):
    print(f"[case] {what} shape={qb.shape} T={T}", flush=True)
    got = run_gpu(qb, kb, vb, mask, T, scale)
    ref = oa.attention(qb, kb, vb, mask, T, scale)
    return assert_parity(got, ref, what)


@pytest.mark.parametrize("form", ["col", "sym", "dense"])
def test_tiny_workload(form):
    w = workloads.WORKLOADS["tiny"]
    qb, kb, vb = workloads.make_workload_qkv(w)
    full_check(qb, kb, vb, om.tile_mask(w.F, w.g, form), w.T, w.scale(), f"tiny-{form}")


@pytest.mark.parametrize("d", [64, 96, 128])
@pytest.mark.parametrize("T", [1, 15, 16, 17, 31, 33, 63, 64, 65, 127, 128, 129, 200, 257])
def test_ragged_tails(d, T):
    F = 3
    B, H = 1, 2
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T * 7 + d)
    mask = np.array([[1, 0, 1], [1, 1, 0], [0, 1, 1]], np.uint8)
    full_check(qb, kb, vb, mask, T, d ** -0.5, f"tails-d{d}-T{T}")


@pytest.mark.parametrize("d", [64, 96, 128])
def test_multi_tile_random_masks(d):
    rng = np.random.default_rng(d)
    B, H, F, T = 2, 3, 5, 300
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=d, dist="frame_shift")
    for trial in range(3):
        mask = (rng.random((F, F)) < 0.45).astype(np.uint8)
        mask[trial, :] = 0  # an empty row: zeros
        full_check(qb, kb, vb, mask, T, d ** -0.5, f"random-d{d}-{trial}")


def test_empty_rows_are_zero():
    B, H, F, T, d = 1, 2, 4, 100, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=3)
    mask = om.tile_mask(F, 1, "col")
    mask[2, :] = 0
    got = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
    assert np.all(got[:, :, 2 * T:3 * T] == 0)


def test_frame_tail_keys_are_used():
    """Spike V on the keys past the last full 64-key tile of each frame: a kernel that
    dropped the ragged frame tail would pass the absolute gate at random inputs but
    not here."""
    B, H, F, T, d = 1, 2, 4, 3600, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=11)
    v = workloads.bf16_bits_to_f32(vb).reshape(B, H, F, T, d)
    v[:, :, :, T - 16:, :] += 8.0
    vb = workloads.f32_to_bf16_bits(v.reshape(B, H, F * T, d))
    mask = om.tile_mask(F, 1, "col")
    got = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
    b, h, s = sample_rows(B, H, F, T, per_frame=8)
    ref = oa.attention_rows(qb, kb, vb, mask, T, d ** -0.5, b, h, s)
    assert_parity(got[b, h, s], ref, "tail-spike")


def test_skipped_tiles_are_never_read():
    """Poison the K/V of frames the mask skips with NaN and 1e30: rows that do not
    keep the poisoned frames must not change by a single bit, which shows those
    tiles are skipped rather than masked. T = 200 leaves a ragged 8-key tail in
    every frame, so a tail load running into the next frame would be caught."""
    B, H, F, T, d = 1, 2, 6, 200, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=5)
    mask = om.tile_mask(F, 2, "col")  # G = {0, 3}
    base = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
    for poisoned_frames in ([4], [1, 5], [2, 4]):
        kp, vp = kb.copy(), vb.copy()
        for j in poisoned_frames:
            kp[:, :, j * T:(j + 1) * T] = 0x7FC0  # NaN
            vp[:, :, j * T:(j + 1) * T] = 0x7149  # about 1e30
        got = run_gpu(qb, kp, vp, mask, T, d ** -0.5)
        clean = [i for i in range(F) if not any(mask[i, j] for j in poisoned_frames)]
        assert clean
        for i in clean:
            assert np.array_equal(got[:, :, i * T:(i + 1) * T], base[:, :, i * T:(i + 1) * T]), i
    ref = oa.attention(qb, kb, vb, mask, T, d ** -0.5)
    assert_parity(base, ref, "poison-base")


def test_dense_control_is_bitwise_all_ones_mask():
    B, H, F, T, d = 1, 3, 4, 300, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=9)
    a = run_gpu(qb, kb, vb, None, T, d ** -0.5, dense=True)
    b = run_gpu(qb, kb, vb, np.ones((F, F), np.uint8), T, d ** -0.5)
    assert np.array_equal(a, b)
    assert_parity(a, oa.attention(qb, kb, vb, np.ones((F, F)), T, d ** -0.5), "dense")


def test_repeat_calls_are_bitwise_equal():
    B, H, F, T, d = 1, 4, 8, 500, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=2)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    mask = om.tile_mask(F, 2, "sym")
    outs = []
    for _ in range(3):
        o = torch.empty_like(q)
        ta.tile_attn_fwd(q, k, v, o, B, H, F, T, d, mask, d ** -0.5)
        outs.append(o)
    torch.cuda.synchronize()
    assert all(torch.equal(outs[0], o) for o in outs[1:])


def test_non_default_stream():
    B, H, F, T, d = 1, 2, 4, 256, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=4)
    mask = om.tile_mask(F, 1, "col")
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = torch.empty_like(q)
        ta.tile_attn_fwd(q, k, v, out, B, H, F, T, d, mask, d ** -0.5, s)
    s.synchronize()
    assert_parity(from_dev(out), oa.attention(qb, kb, vb, mask, T, d ** -0.5), "stream")


def test_output_guard_bands_untouched():
    B, H, F, T, d = 1, 2, 3, 129, 128
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=6)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    n = q.numel()
    guard = 4096
    big = torch.full((n + 2 * guard,), 1.2345, dtype=torch.bfloat16, device="cuda")
    out = big[guard:guard + n].view(B, H, F * T, d)
    mask = om.tile_mask(F, 1, "sym")
    ta.tile_attn_fwd(q, k, v, out, B, H, F, T, d, mask, d ** -0.5)
    torch.cuda.synchronize()
    g = from_dev(big)
    canary = from_dev(torch.tensor([1.2345], dtype=torch.bfloat16))[0]
    assert np.all(g[:guard] == canary) and np.all(g[guard + n:] == canary)
    assert_parity(from_dev(out), oa.attention(qb, kb, vb, mask, T, d ** -0.5), "guard")


@pytest.mark.parametrize("scale", [-0.1, 0.0, 0.35, 2.0])
def test_scale_values(scale):
    B, H, F, T, d = 1, 2, 3, 150, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=12)
    mask = om.tile_mask(F, 1, "col")
    full_check(qb, kb, vb, mask, T, scale, f"scale{scale}")


def test_many_frames_short_tiles():
    """F above 255 exercises 16-bit kept lists; T = 2 puts many frames in one tile."""
    B, H, F, T, d = 1, 1, 300, 2, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=13)
    mask = om.tile_mask(F, 7, "sym")
    full_check(qb, kb, vb, mask, T, d ** -0.5, "F300")


# ---- measured workloads at full size, sampled rows --------------------------------

# Every (workload, mask form, g) the benchmark times (bench.py ALL_CASES), with the
# dense control of each workload.
FULL_CASES = [
    ("29f", "col", 1), ("29f", "sym", 1), ("29f", "dense", 1),
    ("93f", "col", 1), ("93f", "sym", 1), ("93f", "dense", 1),
    ("sweep", "col", 1), ("sweep", "col", 2), ("sweep", "col", 4), ("sweep", "col", 8),
    ("sweep", "sym", 2), ("sweep", "sym", 4), ("sweep", "sym", 8), ("sweep", "dense", 1),
    ("sp_share", "col", 1), ("sp_share", "sym", 1), ("sp_share", "dense", 1),
    ("long", "col", 2), ("long", "sym", 2), ("long", "dense", 2),
    ("93f_d128", "col", 1), ("93f_d128", "sym", 1), ("93f_d128", "dense", 1),
]


@pytest.mark.parametrize("name,form,g", FULL_CASES, ids=[f"{a}-{b}-g{c}" for a, b, c in FULL_CASES])
def test_full_size_sampled(name, form, g):
    w = workloads.WORKLOADS[name]
    print(f"[case] full {name} {form} g={g}", flush=True)
    qb, kb, vb = workload_inputs(name)
    mask = om.tile_mask(w.F, g, form)
    got = run_gpu(qb, kb, vb, mask, w.T, w.scale())
    heads = None if form != "dense" else [0, w.H // 2, w.H - 1]
    b, h, s = sample_rows(w.B, w.H, w.F, w.T, per_frame=2, heads=heads, seed=len(name))
    ref = oa.attention_rows(qb, kb, vb, mask, w.T, w.scale(), b, h, s)
    assert_parity(got[b, h, s], ref, f"{name}-{form}-g{g}")
    # rows of frames that keep nothing do not exist in these masks; outputs are finite
    assert errors(got[:, :, :: max(1, w.T // 7)], np.zeros(1))["finite"]


def test_last_query_block_with_idle_waves():
    """At T = 3600 the last query block of each frame holds 16 rows: two of its four
    waves split the keys of every tile and the other two only help load tiles. No
    wave may overwrite a K buffer that the others still read, nor the LDS that
    carries one wave's softmax state to the other; every row of the last blocks of
    all frames and heads is compared, at a head count that fills the GPU."""
    B, H, F, T, d = 1, 24, 3, 3600, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=21)
    mask = om.tile_mask(F, 1, "col")
    got = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
    rows = np.arange(T - 144, T)
    for h in (0, 7, 23):
        s = np.concatenate([f * T + rows for f in range(F)])
        ref = oa.attention_rows(qb, kb, vb, mask, T, d ** -0.5, np.zeros_like(s), np.full_like(s, h), s)
        assert_parity(got[0, h, s], ref, f"last-block-h{h}")


def test_d64_tail_blocks_full_size():
    """At d = 64 a frame's last query block of 16 rows (T = 3600) runs on two waves
    that split the keys of every tile; every row of the last blocks of all frames is
    compared, at a head count that fills the GPU."""
    B, H, F, T, d = 1, 24, 3, 3600, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=22)
    mask = om.tile_mask(F, 1, "col")
    got = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
    rows = np.arange(T - 144, T)
    for h in (0, 11, 23):
        s = np.concatenate([f * T + rows for f in range(F)])
        ref = oa.attention_rows(qb, kb, vb, mask, T, d ** -0.5, np.zeros_like(s), np.full_like(s, h), s)
        assert_parity(got[0, h, s], ref, f"d64-last-block-h{h}")


@pytest.mark.parametrize("T", [272, 356])
def test_d64_tail_blocks_of_split_frames(T):
    """d = 64 tail blocks (16 or 100 valid rows after a full 256-row block: keys split
    over two waves, or one column block per wave) in the pieces of split heavy frames,
    which write fp32 partials before the merge; every row is compared with the oracle."""
    B, H, F, d = 1, 2, 10, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=23)
    mask = om.tile_mask(F, 1, "sym")
    assert ta.tile_attn_plan(mask)[1] > 0
    full_check(qb, kb, vb, mask, T, d ** -0.5, f"d64-tail-split-T{T}")


SHORT_CASES = [  # (d, T): a last query block of 1 .. 32 rows; T mod 64 sets the last key tile
    (64, 272), (64, 288), (96, 257), (96, 272), (96, 287), (96, 288), (128, 144), (128, 160), (128, 276),
]


@pytest.mark.parametrize("form", ["col", "sym"])
@pytest.mark.parametrize("d,T", SHORT_CASES)
def test_short_last_query_blocks(d, T, form):
    """A segment's last query block with at most 32 valid rows runs (at d = 64 and 96)
    on two waves, each taking one 32-key half of every tile; the second wave's softmax
    state joins the first's through LDS. The last key tile of a frame holds 16, 31 or
    32 keys here, so the second half is empty or partly masked; with sym masks the
    heavy frames are split and the short blocks write partials. At d = 128 the same
    blocks run on one wave. Every row and the log-sum-exp against the oracle."""
    B, H, F = (3, 2, 7) if T == 272 else (1, 3, 7)  # B = 3: shares that cross batch entries
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T * 3 + d)
    mask = om.tile_mask(F, 2, form)
    scale = d ** -0.5
    print(f"[case] short last block B={B} d={d} T={T} {form}", flush=True)
    got, lse = run_gpu_heads(qb, kb, vb, mask, T, scale)
    assert_parity(got, oa.attention(qb, kb, vb, mask, T, scale), f"short-d{d}-T{T}-{form}")
    assert_lse(lse, oa.attention_lse(qb, kb, mask, T, scale), f"short-lse-d{d}-T{T}-{form}")


# ---- split heavy query frames (partial results merged by log-sum-exp) -----------------

@pytest.mark.parametrize("d", [64, 96, 128])
def test_split_heavy_rows(d):
    """The symmetric mask's global query frame keeps every frame: its work is split
    into pieces whose partials are merged; every row is compared with the oracle."""
    B, H, F, T = 2, 3, 10, 150
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=30 + d)
    mask = om.tile_mask(F, 1, "sym")
    assert ta.tile_attn_plan(mask)[1] > 0
    full_check(qb, kb, vb, mask, T, d ** -0.5, f"split-d{d}")


def test_split_random_heavy_masks():
    rng = np.random.default_rng(31)
    B, H, F, T, d = 1, 2, 12, 100, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=31, dist="frame_shift")
    for trial in range(3):
        mask = (rng.random((F, F)) < 0.2).astype(np.uint8)
        mask[3 * trial, :] = 1
        mask[3 * trial + 1, :] = 0  # an empty row next to a split one: zeros
        assert ta.tile_attn_plan(mask)[1] > 0
        full_check(qb, kb, vb, mask, T, d ** -0.5, f"split-random-{trial}")


def test_split_on_two_streams():
    """Each stream has its own workspace for partial results: two split calls queued
    on two streams at once both match the oracle."""
    B, H, F, T, d = 1, 4, 8, 300, 96
    mask = om.tile_mask(F, 1, "sym")
    data = [workloads.make_qkv(B, H, F, T, d, seed=40 + i) for i in range(2)]
    dev = [tuple(to_dev(x) for x in qkv) for qkv in data]
    outs = [torch.empty_like(dq[0]) for dq in dev]
    streams = [torch.cuda.Stream() for _ in range(2)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for rep in range(3):
        for (q, k, v), out, s in zip(dev, outs, streams):
            with torch.cuda.stream(s):
                ta.tile_attn_fwd(q, k, v, out, B, H, F, T, d, mask, d ** -0.5, s)
    torch.cuda.synchronize()
    for (qb, kb, vb), out in zip(data, outs):
        assert_parity(from_dev(out), oa.attention(qb, kb, vb, mask, T, d ** -0.5), "split-streams")


def test_split_workspace_grows():
    """A larger split call after a smaller one grows the workspace; the smaller call
    afterwards still matches."""
    d = 64
    cases = [(1, 2, 6, 100), (2, 4, 9, 260), (1, 2, 6, 100)]
    for B, H, F, T in cases:
        qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=B * 100 + F)
        mask = om.tile_mask(F, 1, "sym")
        full_check(qb, kb, vb, mask, T, d ** -0.5, f"split-grow-{B}x{H}x{F}x{T}")


# ---- one mask per head and the row log-sum-exp ----------------------------------------

LSE_MAX_ABS = 5e-3  # natural-log units; the GPU sums the bf16-rounded weights


def run_gpu_heads(qb, kb, vb, masks, T, scale):
    B, H, S, d = qb.shape
    F = S // T
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    out = torch.empty_like(q)
    lse = torch.full((B, H, S), 12345.0, dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, masks, scale, lse,
                           torch.cuda.current_stream())
    torch.cuda.synchronize()
    return from_dev(out), lse.cpu().numpy().astype(np.float64)


def assert_lse(got, ref, what):
    empty = np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), empty), f"{what}: -inf rows differ"
    err = np.abs(got[~empty] - ref[~empty])
    print(f"[lse] {what} max abs {err.max() if err.size else 0.0:.2e}", flush=True)
    assert err.size == 0 or err.max() <= LSE_MAX_ABS, f"{what}: lse max abs {err.max()}"


def _head_masks(F):
    rng = np.random.default_rng(F)
    rand = (rng.random((F, F)) < 0.4).astype(np.uint8)
    rand[1, :] = 0
    return np.stack([np.ones((F, F), np.uint8), om.tile_mask(F, 1, "col"),
                     om.tile_mask(F, 1, "sym"), rand])


@pytest.mark.parametrize("d", [64, 96, 128])
def test_per_head_masks_and_lse(d):
    B, H, F, T = 2, 4, 7, 130
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=50 + d, dist="frame_shift")
    masks = _head_masks(F)
    got, lse = run_gpu_heads(qb, kb, vb, masks, T, d ** -0.5)
    assert_parity(got, oa.attention(qb, kb, vb, masks, T, d ** -0.5), f"heads-d{d}")
    assert_lse(lse, oa.attention_lse(qb, kb, masks, T, d ** -0.5), f"heads-d{d}")


def test_shared_mask_heads_matches_tile_attn_fwd_bitwise():
    B, H, F, T, d = 1, 3, 6, 200, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=55)
    for form in ("col", "sym"):
        mask = om.tile_mask(F, 2, form)
        a = run_gpu(qb, kb, vb, mask, T, d ** -0.5)
        b, lse = run_gpu_heads(qb, kb, vb, mask, T, d ** -0.5)
        assert np.array_equal(a, b), form
        assert_lse(lse, oa.attention_lse(qb, kb, mask, T, d ** -0.5), f"shared-{form}")


@pytest.mark.parametrize("scale", [-0.1, 0.0, 0.35])
def test_lse_scales(scale):
    B, H, F, T, d = 1, 2, 5, 70, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=56)
    masks = np.stack([om.tile_mask(F, 1, "sym"), om.tile_mask(F, 2, "col")])
    got, lse = run_gpu_heads(qb, kb, vb, masks, T, scale)
    assert_parity(got, oa.attention(qb, kb, vb, masks, T, scale), f"lse-scale{scale}")
    assert_lse(lse, oa.attention_lse(qb, kb, masks, T, scale), f"lse-scale{scale}")


def test_per_head_masks_full_size_sampled():
    """93-frame 720p shape with a different k:(F-k) pattern per head (col and sym, g = 1,
    2, 4, 8): sampled rows of every head, and the log-sum-exp of two heads in full."""
    w = workloads.WORKLOADS["93f"]
    qb, kb, vb = workload_inputs("93f")
    masks = np.stack([om.tile_mask(w.F, [1, 2, 4, 8][h % 4], "col" if h % 2 else "sym")
                      for h in range(w.H)])
    got, lse = run_gpu_heads(qb, kb, vb, masks, w.T, w.scale())
    b, h, s = sample_rows(w.B, w.H, w.F, w.T, per_frame=2, seed=57)
    ref = oa.attention_rows(qb, kb, vb, masks, w.T, w.scale(), b, h, s)
    assert_parity(got[b, h, s], ref, "heads-93f")
    for hh in (0, 5):
        ref_lse = oa.attention_lse(qb[:, hh:hh + 1], kb[:, hh:hh + 1], masks[hh], w.T, w.scale())
        assert_lse(lse[:, hh:hh + 1], ref_lse, f"heads-93f-lse-h{hh}")


def test_hip_graph_capture_and_replay():
    """A warmed-up call (its work list uploaded and its workspace sized on the capture
    stream) records into a HIP graph: forward with split rows (attention kernel and
    merge) and the gradients. Several replays, with eager work and synchronisation
    between them, each equal the eager result bit for bit."""
    B, H, F, T, d = 1, 2, 10, 100, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=120)
    rng = np.random.default_rng(121)
    gb = workloads.f32_to_bf16_bits(rng.standard_normal(qb.shape).astype(np.float32))
    mask = om.tile_mask(F, 1, "sym")
    assert ta.tile_attn_plan(mask)[1] > 0 and ta.tile_attn_plan(mask.T.copy())[1] > 0  # splits on both sides
    scale = d ** -0.5
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        q, k, v, g = (to_dev(x) for x in (qb, kb, vb, gb))
        out = torch.empty_like(q)
        lse = torch.empty((B, H, F * T), dtype=torch.float32, device="cuda")
        grads = [torch.empty_like(q) for _ in range(3)]

    def step():
        ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, mask, scale, lse, s)
        ta.tile_attn_bwd(q, k, v, out, g, lse, *grads, B, H, F, T, d, mask, scale, s)

    with torch.cuda.stream(s):
        for _ in range(2):
            step()
    s.synchronize()
    eager = [from_dev(x) for x in [out] + grads]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        step()
    for rep in range(3):
        for x in [out] + grads:
            x.fill_(float("nan"))  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, e in zip([from_dev(x) for x in [out] + grads], eager):
            assert np.array_equal(a, e), rep
    assert_parity(eager[0], oa.attention(qb, kb, vb, mask, T, scale), "graph-fwd")


def test_max_frames():
    """F = TA_MAX_FRAMES (1024) with tiny frames: a random sparse mask with some full
    rows (split) and empty rows, through the forward."""
    B, H, F, T, d = 1, 2, 1024, 3, 64
    rng = np.random.default_rng(130)
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=130)
    mask = (rng.random((F, F)) < 0.01).astype(np.uint8)
    mask[::97, :] = 1
    mask[5::211, :] = 0
    full_check(qb, kb, vb, mask, T, d ** -0.5, "max-frames")


# ---- the ragged last round of an XCD run in parts over the kept tiles ----------------

PART_CASES = [  # (B, H, F, T, d, g, form): each XCD's last round is cut into parts
    (1, 16, 17, 500, 64, 1, "col"),
    (1, 12, 20, 700, 96, 2, "col"),
    (1, 32, 6, 700, 96, 1, "sym"),
    (1, 8, 11, 700, 128, 1, "col"),
    # 16-row last query blocks: at d = 64 on two waves, last in each share, no parts;
    # at d = 128 on one wave, among the parts
    (1, 32, 6, 528, 64, 1, "col"),
    (1, 20, 6, 528, 128, 1, "col"),
]


@pytest.mark.parametrize("B,H,F,T,d,g,form", PART_CASES)
def test_ragged_round_in_parts(B, H, F, T, d, g, form):
    """Launches whose XCDs would end on a ragged round of whole query blocks run that
    round's blocks in parts over the kept tiles (merged by log-sum-exp; the host check
    in tests/test_schedule.py confirms these shapes are cut, all but the d = 64 one with
    16-row last blocks, which runs those blocks last instead). Sampled rows of every
    frame and head, and the log-sum-exp of two heads, against the oracle."""
    print(f"[case] parts B={B} H={H} F={F} T={T} d={d} {form} g={g}", flush=True)
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=F * T + d)
    mask = om.tile_mask(F, g, form)
    scale = d ** -0.5
    got, lse = run_gpu_heads(qb, kb, vb, mask, T, scale)
    b, h, s = sample_rows(B, H, F, T, per_frame=6, seed=T)
    assert_parity(got[b, h, s], oa.attention_rows(qb, kb, vb, mask, T, scale, b, h, s), "parts")
    for hh in (0, H - 1):
        ref = oa.attention_lse(qb[:, hh:hh + 1], kb[:, hh:hh + 1], mask, T, scale)
        assert_lse(lse[:, hh:hh + 1], ref, f"parts-lse-h{hh}")
    # the plain entry point takes the same schedule: same bits
    assert np.array_equal(run_gpu(qb, kb, vb, mask, T, scale), got)


def test_ragged_round_in_parts_with_empty_frames():
    """Query frames that keep nothing (every seventh) in a launch whose XCDs end on a
    ragged round cut into parts (tests/test_schedule.py covers the same shape): a
    block with rows and no kept tile still runs, writing zeros and a -inf
    log-sum-exp, wherever it falls in the schedule."""
    B, H, F, T, d = 1, 12, 20, 700, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=4242)
    mask = om.tile_mask(F, 2, "col")
    empty = list(range(6, F, 7))
    mask[empty, :] = 0
    scale = d ** -0.5
    print(f"[case] parts with empty frames {empty}", flush=True)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((B, H, F * T), 12345.0, dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, mask, scale, lse, torch.cuda.current_stream())
    torch.cuda.synchronize()
    got, lse = from_dev(out), lse.cpu().numpy().astype(np.float64)
    for f in empty:
        rows = slice(f * T, (f + 1) * T)
        assert np.all(got[:, :, rows] == 0), f
        assert np.all(np.isneginf(lse[:, :, rows])), f
    b, h, srows = sample_rows(B, H, F, T, per_frame=4, seed=7)
    assert_parity(got[b, h, srows], oa.attention_rows(qb, kb, vb, mask, T, scale, b, h, srows), "parts-empty")
