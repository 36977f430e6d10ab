"""Parity of the MM-DiT form (tile_attn_fwd_mmdit: dense text prefix before the
tile-sparse video) with the float64 oracle, through the C ABI."""
import numpy as np
import pytest

import workloads
from oracle import attention as oa
from oracle import masks as om
from oracle import mmdit as ommd
from tests.gpu_helpers import assert_parity, from_dev, to_dev, workload_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402

LSE_MAX_ABS = 5e-3


def run_mmdit(qb, kb, vb, masks, T, P, scale, with_lse=True):
    B, H, S, d = qb.shape
    F = (S - P) // T
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((B, H, S), 12345.0, dtype=torch.float32, device="cuda") if with_lse else None
    ta.tile_attn_fwd_mmdit(q, k, v, out, B, H, F, T, P, d, masks, scale, lse,
                           torch.cuda.current_stream())
    torch.cuda.synchronize()
    return from_dev(out), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def assert_lse(got, ref, what):
    assert np.array_equal(np.isneginf(got), np.isneginf(ref)), what
    ok = ~np.isneginf(ref)
    err = np.abs(got[ok] - ref[ok]).max()
    print(f"[lse] {what} max abs {err:.2e}", flush=True)
    assert err <= LSE_MAX_ABS, f"{what}: lse max abs {err}"


def _masks(F, H, seed):
    rng = np.random.default_rng(seed)
    ms = (rng.random((H, F, F)) < 0.4).astype(np.uint8)
    ms[0, 1, :] = 0  # a video frame that keeps no video frame still attends the text
    return ms


@pytest.mark.parametrize("d", [64, 96, 128])
@pytest.mark.parametrize("P", [1, 17, 64, 226, 300])
def test_mmdit_small(d, P):
    B, H, F, T = 2, 3, 4, 130
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=P + d, dist="frame_shift", prefix=P)
    masks = _masks(F, H, P)
    print(f"[case] mmdit d={d} P={P}", flush=True)
    got, lse = run_mmdit(qb, kb, vb, masks, T, P, d ** -0.5)
    assert_parity(got, ommd.attention_mmdit(qb, kb, vb, masks, T, P, d ** -0.5), f"mmdit-d{d}-P{P}")
    assert_lse(lse, ommd.attention_mmdit_lse(qb, kb, masks, T, P, d ** -0.5), f"mmdit-d{d}-P{P}")


@pytest.mark.parametrize("T,P", [(1, 3), (64, 1), (65, 200), (100, 1000), (257, 5)])
def test_mmdit_segment_lengths(T, P):
    """Text longer or shorter than a frame, one-token frames, several query blocks of
    text (P = 1000) and ragged tails on both sides."""
    B, H, F, d = 1, 2, 3, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T * 7 + P, prefix=P)
    mask = om.tile_mask(F, 1, "sym")
    got, lse = run_mmdit(qb, kb, vb, mask, T, P, 0.125)
    assert_parity(got, ommd.attention_mmdit(qb, kb, vb, mask, T, P, 0.125), f"seg-T{T}-P{P}")
    assert_lse(lse, ommd.attention_mmdit_lse(qb, kb, mask, T, P, 0.125), f"seg-T{T}-P{P}")


def test_mmdit_without_text_matches_heads_bitwise():
    B, H, F, T, d = 1, 3, 6, 200, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=77)
    masks = np.stack([om.tile_mask(F, 2, "col"), om.tile_mask(F, 1, "sym"), np.eye(F, dtype=np.uint8)])
    got, lse = run_mmdit(qb, kb, vb, masks, T, 0, d ** -0.5)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    out = torch.empty_like(q)
    lse2 = torch.empty((B, H, F * T), dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, masks, d ** -0.5, lse2, None)
    torch.cuda.synchronize()
    assert np.array_equal(got, from_dev(out))
    assert np.array_equal(lse, lse2.cpu().numpy().astype(np.float64))
    assert_parity(got, oa.attention(qb, kb, vb, masks, T, d ** -0.5), "mmdit-P0")


def test_mmdit_skipped_video_frames_are_never_read():
    """NaN-poison the k, v of video frames the mask skips for some rows: those rows,
    and no others, may change; the text is always read, so poisoning it must change
    every row."""
    B, H, F, T, P, d = 1, 2, 5, 150, 40, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=78, prefix=P)
    mask = om.tile_mask(F, 2, "col")  # G = {0, 3}
    base, _ = run_mmdit(qb, kb, vb, mask, T, P, 0.125, with_lse=False)
    kp, vp = kb.copy(), vb.copy()
    j = 4
    kp[:, :, P + j * T:P + (j + 1) * T] = 0x7FC0
    vp[:, :, P + j * T:P + (j + 1) * T] = 0x7FC0
    got, _ = run_mmdit(qb, kp, vp, mask, T, P, 0.125, with_lse=False)
    for i in range(F):
        rows = slice(P + i * T, P + (i + 1) * T)
        if not mask[i, j]:
            assert np.array_equal(got[:, :, rows], base[:, :, rows]), i
    assert not np.array_equal(got[:, :, :P], base[:, :, :P])  # text rows see every frame
    assert_parity(base, ommd.attention_mmdit(qb, kb, vb, mask, T, P, 0.125), "mmdit-poison-base")


@pytest.mark.parametrize("k", [1, 2, 3, 4, 6, 12, 0])
def test_mmdit_cog_shape_sampled(k):
    """CogVideoX-5B shape (App. E reading: 13 latent frames x 1350 tokens, 226 text
    tokens, 48 heads of 64), sym masks with k global frames (labels 12, 6, 4, 3, 2, 1
    of tab:cog_kernel; k = 0 stands for the dense control, every tile kept): every text
    row and sampled video rows of three heads."""
    w = workloads.WORKLOADS["cog"]
    qb, kb, vb = workload_inputs("cog")
    mask = om.tile_mask(w.F, k, "sym") if k else np.ones((w.F, w.F), np.uint8)
    print(f"[case] cog k={k}", flush=True)
    got, lse = run_mmdit(qb, kb, vb, mask, w.T, w.prefix, w.scale())
    rng = np.random.default_rng(k)
    rows = []
    for h in (0, 17, w.H - 1):
        rows += [(0, h, s) for s in range(w.prefix)]
        for f in range(w.F):
            for r in {0, w.T - 1, int(rng.integers(0, w.T))}:
                rows.append((0, h, w.prefix + f * w.T + r))
    b, h, s = (np.array(x) for x in zip(*rows))
    ref = ommd.attention_mmdit_rows(qb, kb, vb, mask, w.T, w.prefix, w.scale(), b, h, s)
    assert_parity(got[b, h, s], ref, f"cog-k{k}")
    hh = 17
    ref_lse = ommd.attention_mmdit_lse(qb[:, hh:hh + 1], kb[:, hh:hh + 1], mask, w.T, w.prefix, w.scale())
    assert_lse(lse[:, hh:hh + 1], ref_lse, f"cog-k{k}-lse")


def test_mmdit_ragged_round_in_parts():
    """An MM-DiT launch (12 heads of 64, 9 frames x 1350 tokens, 226 text tokens, sym
    g=1) whose XCDs end on a ragged round: that round's query blocks, text blocks
    included, run in parts over their kept tiles (tests/test_schedule.py confirms the
    cut). Every text row and sampled video rows of two heads, and their log-sum-exp."""
    B, H, F, T, P, d = 1, 12, 9, 1350, 226, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=P + F, prefix=P)
    mask = om.tile_mask(F, 1, "sym")
    scale = d ** -0.5
    print(f"[case] mmdit parts H={H} F={F} T={T} P={P} d={d}", flush=True)
    got, lse = run_mmdit(qb, kb, vb, mask, T, P, scale)
    rng = np.random.default_rng(F)
    rows = []
    for h in (0, H - 1):
        rows += [(0, h, s) for s in range(P)]
        for f in range(F):
            for r in {0, T - 1, 1279, int(rng.integers(0, T))}:
                rows.append((0, h, P + f * T + r))
    b, h, s = (np.array(x) for x in zip(*rows))
    ref = ommd.attention_mmdit_rows(qb, kb, vb, mask, T, P, scale, b, h, s)
    assert_parity(got[b, h, s], ref, "mmdit-parts")
    for hh in (0, H - 1):
        ref_lse = ommd.attention_mmdit_lse(qb[:, hh:hh + 1], kb[:, hh:hh + 1], mask, T, P, scale)
        assert_lse(lse[:, hh:hh + 1], ref_lse, f"mmdit-parts-lse-h{hh}")


@pytest.mark.parametrize("T,P", [(272, 20), (528, 3)])
def test_mmdit_short_blocks_in_work_loop(T, P):
    """Query blocks of at most 32 rows (the whole text, and each frame's 16-row last
    block) in the persistent work loop of a split MM-DiT plan at d = 64: their two
    waves pass one wave's softmax state to the other through the LDS that the next
    unit's tile loads then reuse. Every row and the log-sum-exp against the oracle."""
    B, H, F, d = 1, 4, 10, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=T + P, prefix=P)
    mask = om.tile_mask(F, 1, "sym")
    aug = np.ones((F + 1, F + 1), np.uint8)
    aug[:F, :F] = mask
    assert ta.tile_attn_plan(aug)[1] > 0  # split frames: the persistent loop runs
    print(f"[case] mmdit short blocks T={T} P={P}", flush=True)
    got, lse = run_mmdit(qb, kb, vb, mask, T, P, d ** -0.5)
    assert_parity(got, ommd.attention_mmdit(qb, kb, vb, mask, T, P, d ** -0.5), f"short-T{T}-P{P}")
    assert_lse(lse, ommd.attention_mmdit_lse(qb, kb, mask, T, P, d ** -0.5), f"short-T{T}-P{P}")


def test_mmdit_work_queue_in_graph_and_between_calls():
    """The MM-DiT form at d = 64 with split frames runs the kernel's persistent work
    loop, whose queue counters (per stream) every launch must leave at zero: eager
    calls of two shapes in turn on one stream, then a captured graph replayed several
    times with eager calls in between, all equal their first eager result bit for bit."""
    d, P = 64, 77
    shapes = [(1, 6, 11, 300), (2, 3, 12, 130)]
    inputs = []
    for i, (B, H, F, T) in enumerate(shapes):
        qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=900 + i, prefix=P)
        mask = om.tile_mask(F, 1, "sym")
        aug = np.ones((F + 1, F + 1), np.uint8)  # the text segment's row and column kept
        aug[:F, :F] = mask
        assert ta.tile_attn_plan(aug)[1] > 0  # split frames: the persistent loop runs
        inputs.append((qb, kb, vb, mask, T))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    dev = []
    with torch.cuda.stream(s):
        for qb, kb, vb, masks, T in inputs:
            q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
            dev.append((q, k, v, torch.empty_like(q), masks, T))

    def call(i):
        q, k, v, out, masks, T = dev[i]
        B, H, S, _ = q.shape
        ta.tile_attn_fwd_mmdit(q, k, v, out, B, H, (S - P) // T, T, P, d, masks, d ** -0.5, None, s)

    with torch.cuda.stream(s):
        for _ in range(3):
            call(0)
            call(1)
    s.synchronize()
    first = [from_dev(x[3]) for x in dev]
    for i, (qb, kb, vb, masks, T) in enumerate(inputs):
        assert_parity(first[i], ommd.attention_mmdit(qb, kb, vb, masks, T, P, d ** -0.5), f"queue-{i}")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        call(0)
    for rep in range(3):
        dev[0][3].fill_(float("nan"))
        with torch.cuda.stream(s):
            call(1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(dev[0][3]), first[0]), rep
        assert np.array_equal(from_dev(dev[1][3]), first[1]), rep
