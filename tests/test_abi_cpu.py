"""Host-side checks of the C ABI that need no GPU: exports, mask builder and
compaction parity with the oracle, and argument errors (returned before any
HIP call, so nothing is enqueued)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2502_06155_amd as ta
from oracle import attention as oa
from oracle import masks as om
from paper_2502_06155_amd._lib import lib
from tests.conftest import ROOT


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "tile_attn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert "tile_attn_fwd" in names and "dense_attn_fwd" in names
    for name in names:
        assert hasattr(lib, name), f"{name} declared in tile_attn.h but not exported"


@pytest.mark.parametrize("form", ["col", "sym", "dense"])
def test_make_mask_matches_oracle(form):
    for F in list(range(1, 50)) + [64, 100, 255, 1024]:
        ks = range(0, F + 1) if F <= 49 else (0, 1, 2, 7, F)
        for k in ks:
            got = ta.tile_attn_make_mask(F, k, form)
            assert np.array_equal(got, om.tile_mask(F, k, form)), (F, k, form)


def test_compact_matches_oracle_kept_frames():
    rng = np.random.default_rng(0)
    masks = [om.tile_mask(24, 1, "col"), om.tile_mask(24, 4, "sym"), np.zeros((5, 5), np.uint8)]
    masks += [(rng.random((F, F)) < p).astype(np.uint8) for F in (1, 2, 7, 33) for p in (0.1, 0.5, 0.9)]
    for M in masks:
        F = M.shape[0]
        row_ptr, cols, order = ta.tile_attn_compact(M)
        assert row_ptr[0] == 0 and row_ptr[-1] == om.nnz(M) == len(cols)
        for i in range(F):
            assert list(cols[row_ptr[i]:row_ptr[i + 1]]) == oa.kept_frames(M, i)
        counts = np.diff(row_ptr)
        assert sorted(order.tolist()) == list(range(F))
        assert all(counts[order[a]] >= counts[order[a + 1]] for a in range(F - 1))
        # ties keep frame order
        for a in range(F - 1):
            if counts[order[a]] == counts[order[a + 1]]:
                assert order[a] < order[a + 1]


def test_compact_nonzero_bytes_count_as_kept():
    M = np.array([[0, 7], [255, 1]], dtype=np.uint8)
    row_ptr, cols, _ = ta.tile_attn_compact(M)
    assert row_ptr.tolist() == [0, 1, 3] and cols.tolist() == [1, 0, 1]


def _fwd(q=16, k=32, v=48, out=4096, B=1, H=1, F=2, T=8, d=64, mask=None, scale=0.125):
    m = np.ones((F, F), np.uint8) if mask is None else mask
    mp = m.ctypes.data if m is not False else None
    return lib.tile_attn_fwd(q, k, v, out, B, H, F, T, d, mp, scale, None)


def test_argument_errors_before_any_gpu_call():
    assert _fwd(q=None) == 1
    assert _fwd(out=None) == 1
    assert _fwd(mask=False) == 1
    assert _fwd(B=0) == 2 and _fwd(H=-1) == 2 and _fwd(F=0) == 2 and _fwd(T=0) == 2
    assert _fwd(F=1025, mask=np.ones((1025, 1025), np.uint8)) == 2
    assert _fwd(F=2, T=2 ** 30 + 1) == 2  # F*T > 2^31 - 1
    assert _fwd(B=4096, H=4096, F=4, T=128, mask=np.ones((4, 4), np.uint8)) == 2  # grid limit
    for d in (0, 32, 80, 160, 256):
        assert _fwd(d=d) == 3
    assert _fwd(q=18) == 5 and _fwd(out=4100) == 5
    assert _fwd(scale=float("nan")) == 6 and _fwd(scale=float("inf")) == 6
    assert _fwd(out=16) == 7 and _fwd(out=32 + 16) == 7
    msg = lib.tile_attn_last_error().decode()
    assert "overlap" in msg
    assert lib.dense_attn_fwd(16, 32, 48, 4096, 1, 1, 2, 8, 72, 0.1, None) == 3


def test_make_mask_errors():
    buf = np.zeros(16, np.uint8)
    assert lib.tile_attn_make_mask(4, 5, 0, buf.ctypes.data) == 4
    assert lib.tile_attn_make_mask(4, -1, 0, buf.ctypes.data) == 4
    assert lib.tile_attn_make_mask(4, 1, 3, buf.ctypes.data) == 4
    assert lib.tile_attn_make_mask(0, 0, 0, buf.ctypes.data) == 2
    assert lib.tile_attn_make_mask(4, 1, 0, None) == 1
    with pytest.raises(ta.TileAttnError):
        ta.tile_attn_make_mask(4, 9, "col")


def test_status_strings():
    for s in range(9):
        assert lib.tile_attn_status_string(s)
    assert lib.tile_attn_status_string(99) == b"unknown status"


def _plan_invariants(M, items, n_slots):
    F = M.shape[0]
    counts = M.astype(bool).sum(axis=1)
    row_ptr = np.concatenate([[0], np.cumsum(counts)])
    # every kept entry of every row covered exactly once, pieces contiguous and in order
    by_frame = {}
    for fr, beg, cnt, slot in items:
        by_frame.setdefault(int(fr), []).append((int(slot), int(beg), int(cnt)))
    assert sorted(by_frame) == list(range(F))
    used = set()
    for fr, pieces in by_frame.items():
        pieces.sort()
        if len(pieces) == 1:
            slot, beg, cnt = pieces[0]
            assert slot == -1 and beg == row_ptr[fr] and cnt == counts[fr]
        else:
            assert all(s >= 0 for s, _, _ in pieces)
            pos = row_ptr[fr]
            for s, beg, cnt in pieces:
                assert beg == pos and cnt >= 1
                pos += cnt
                used.add(s)
            assert pos == row_ptr[fr + 1]
    assert used == set(range(n_slots))
    # longest items first
    assert all(items[i, 2] >= items[i + 1, 2] for i in range(len(items) - 1))


def test_plan_splits_only_heavy_rows():
    M = om.tile_mask(24, 1, "sym")  # row 0 keeps 24 frames, the others 2; mean 70/24 -> 3
    items, n_slots = ta.tile_attn_plan(M)
    _plan_invariants(M, items, n_slots)
    heavy = items[items[:, 0] == 0]
    assert n_slots == 8 and len(heavy) == 8 and all(heavy[:, 2] == 3)
    for form, g in (("col", 1), ("col", 8), ("dense", 0), ("sym", 8)):
        M = om.tile_mask(24, g, form)
        items, n_slots = ta.tile_attn_plan(M)
        _plan_invariants(M, items, n_slots)
        assert n_slots == 0 and len(items) == 24


def test_plan_random_masks_and_caps():
    rng = np.random.default_rng(7)
    for F in (1, 2, 5, 33, 100):
        for p in (0.05, 0.3, 0.9):
            M = (rng.random((F, F)) < p).astype(np.uint8)
            M[rng.integers(0, F)] = 1  # one dense row
            items, n_slots = ta.tile_attn_plan(M)
            _plan_invariants(M, items, n_slots)
            assert all(len(items[items[:, 0] == f]) <= 32 for f in range(F))
    M = np.ones((4, 4), np.uint8)
    buf = np.zeros(4, np.int32)
    n, s = ctypes.c_int(0), ctypes.c_int(0)
    assert lib.tile_attn_plan(M.ctypes.data, 4, buf.ctypes.data, 1, ctypes.byref(n), ctypes.byref(s)) == 2
    assert n.value == 4


def _heads(q=1 << 12, k=2 << 12, v=3 << 12, out=4 << 12, B=1, H=2, F=2, T=8, d=64, masks=None,
           n=None, lse=None,
           scale=0.125):
    m = np.ones((H, F, F), np.uint8) if masks is None else masks
    nm = m.size // (F * F) if n is None else n
    return lib.tile_attn_fwd_heads(q, k, v, out, B, H, F, T, d, m.ctypes.data, nm, scale, lse, None)


def test_heads_argument_errors_before_any_gpu_call():
    assert _heads(n=3) == 4 and _heads(n=0) == 4  # n_masks neither 1 nor H
    assert _heads(q=1 << 13, k=2 << 13, v=3 << 13, out=4 << 13, masks=np.ones((1, 2, 2), np.uint8), n=2, H=3) == 4
    assert lib.tile_attn_fwd_heads(1 << 12, 2 << 12, 3 << 12, 4 << 12, 1, 2, 2, 8, 64, None, 2, 0.1,
                                   None, None) == 1
    assert _heads(lse=1 << 20 | 2) == 5  # misaligned lse
    assert _heads(lse=(2 << 12) + 64) == 7  # lse overlaps k
    assert "overlap" in lib.tile_attn_last_error().decode()
    assert _heads(d=80) == 3 and _heads(B=0) == 2


def _bwd(q=1 << 12, k=2 << 12, v=3 << 12, out=4 << 12, dout=5 << 12, lse=6 << 12, dq=7 << 12,
         dk=8 << 12, dv=9 << 12, B=1, H=2, F=2, T=8, d=64, masks=None, n=None, scale=0.125):
    m = np.ones((H, F, F), np.uint8) if masks is None else masks
    nm = m.size // (F * F) if n is None else n
    return lib.tile_attn_bwd(q, k, v, out, dout, lse, dq, dk, dv, B, H, F, T, d, m.ctypes.data, nm,
                             scale, None)


def test_bwd_argument_errors_before_any_gpu_call():
    # every tensor of B=1, H=2, F=2, T=8, d=64 spans 4 KiB: the defaults are disjoint
    assert _bwd(dout=None) == 1 and _bwd(lse=None) == 1 and _bwd(dv=None) == 1
    assert lib.tile_attn_bwd(1 << 12, 2 << 12, 3 << 12, 4 << 12, 5 << 12, 6 << 12, 7 << 12,
                             8 << 12, 9 << 12, 1, 2, 2, 8, 64, None, 2, 0.1, None) == 1
    assert _bwd(n=3) == 4 and _bwd(n=0) == 4
    assert _bwd(d=80) == 3 and _bwd(B=0) == 2 and _bwd(F=2000) == 2
    assert _bwd(scale=float("inf")) == 6
    assert _bwd(dk=(8 << 12) + 8) == 5 and _bwd(dout=(5 << 12) + 2) == 5
    assert _bwd(lse=(6 << 12) + 2) == 5
    assert _bwd(dq=(1 << 12) + 64) == 7  # dq overlaps q
    assert _bwd(dk=(9 << 12) - 1024) == 7  # dk overlaps dv
    assert "each other" in lib.tile_attn_last_error().decode()
    assert _bwd(dv=(5 << 12) + 16) == 7  # dv overlaps dout
    assert _bwd(lse=(7 << 12) + 64) == 7  # dq overlaps lse
    assert "lse" in lib.tile_attn_last_error().decode()


def _mmdit(q=1 << 13, k=2 << 13, v=3 << 13, out=4 << 13, B=1, H=2, F=2, T=8, P=5, d=64, masks=None,
           n=None, lse=None, scale=0.125):
    # each tensor of B=1, H=2, P + F*T = 21 tokens, d=64 spans 5376 bytes < 8 KiB
    m = np.ones((H, F, F), np.uint8) if masks is None else masks
    nm = m.size // (F * F) if n is None else n
    return lib.tile_attn_fwd_mmdit(q, k, v, out, B, H, F, T, P, d, m.ctypes.data, nm, scale, lse, None)


def test_mmdit_argument_errors_before_any_gpu_call():
    assert _mmdit(P=-1) == 2 and _mmdit(B=0) == 2 and _mmdit(d=80) == 3
    assert _mmdit(n=3) == 4
    assert lib.tile_attn_fwd_mmdit(1 << 13, 2 << 13, 3 << 13, 4 << 13, 1, 2, 2, 8, 5, 64, None, 2, 0.1,
                                   None, None) == 1
    assert _mmdit(out=(3 << 13) + 4096) == 7  # out overlaps v within P + F*T tokens
    assert _mmdit(lse=(1 << 20) | 2) == 5
    assert _mmdit(lse=(2 << 13) + 5000) == 7  # lse overlaps k's last rows
    assert _mmdit(T=2 ** 30, F=2, P=2 ** 30) == 2  # P + F*T overflows


def test_bwd_mmdit_argument_errors_before_any_gpu_call():
    # B=1, H=2, F=2, T=8, P=5, d=64: 21 tokens, 5376 bytes per tensor; pointers 8 KiB apart
    base = dict(q=1 << 13, k=2 << 13, v=3 << 13, out=4 << 13, dout=5 << 13, lse=6 << 13, dq=7 << 13,
                dk=8 << 13, dv=9 << 13)

    def call(P=5, d=64, n=2, **kw):
        a = dict(base, **kw)
        m = np.ones((2, 2, 2), np.uint8)
        return lib.tile_attn_bwd_mmdit(a["q"], a["k"], a["v"], a["out"], a["dout"], a["lse"], a["dq"],
                                       a["dk"], a["dv"], 1, 2, 2, 8, P, d, m.ctypes.data, n, 0.1, None)

    assert call(P=-1) == 2 and call(d=80) == 3 and call(n=3) == 4
    assert call(dout=None) == 1
    assert call(dq=(1 << 13) + 4096) == 7  # dq overlaps q over P + F*T tokens
    assert call(dk=(9 << 13) - 4096) == 7  # dk overlaps dv


def test_torch_wrappers_reject_mismatched_tensors_before_launch():
    """The torch wrappers check k, v and out against q's shape before anything reaches
    the library (on CPU tensors the shape check fires first; nothing is launched)."""
    torch = pytest.importorskip("torch")
    q = torch.zeros(1, 2, 4 * 8, 64, dtype=torch.bfloat16)
    small = torch.zeros(1, 2, 4 * 8 - 8, 64, dtype=torch.bfloat16)
    mask = np.ones((4, 4), np.uint8)
    for args in ((q, small, q), (q, q, small)):
        with pytest.raises(ValueError, match="shape"):
            ta.tile_attn(*args, mask, T=8)
        with pytest.raises(ValueError, match="shape"):
            ta.dense_attn(*args, T=8)
    with pytest.raises(ValueError, match="shape"):
        ta.tile_attn(q, q, q, mask, T=8, out=small)
    with pytest.raises(ValueError, match="GPU"):
        ta.tile_attn(q, q, q, mask, T=8)


def test_bf16_rounding_of_the_input_recipe():
    """workloads.f32_to_bf16_bits rounds to nearest, ties to even (torch's float32 ->
    bfloat16 conversion), across the pieces it works through."""
    torch = pytest.importorskip("torch")
    import workloads

    rng = np.random.default_rng(5)
    x = rng.standard_normal((1 << 20) + 77).astype(np.float32) * 10.0 ** rng.integers(-6, 6, (1 << 20) + 77)
    x = x.astype(np.float32)
    ties = (np.arange(1, 2001, dtype=np.uint32) << 16 | 0x8000).view(np.float32)  # exact halfway values
    x = np.concatenate([x, ties, -ties, np.float32([0.0, -0.0, 1.0, 3.4e38])])
    got = workloads.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)
    with pytest.raises(ValueError):
        workloads.f32_to_bf16_bits(np.float32([1.0, np.nan]))


def test_noalloc_rejects_a_plan_beyond_its_scratch_before_any_gpu_call():
    """tile_attn_fwd_heads_noalloc refuses a plan of more than TA_NOALLOC_PLAN_WORDS words
    before anything is enqueued (the buffers are fake addresses that nothing touches)."""
    B, H, F, T, d = 1, 128, 128, 64, 64
    masks = np.ones((H, F, F), np.uint8)  # 5 * 128 * 128 item words + 128^3 kept entries
    fake = 1 << 40
    with pytest.raises(ta.TileAttnError, match="static scratch"):
        ta.tile_attn_fwd_heads_noalloc(fake, fake + (1 << 30), fake + (2 << 30), fake + (3 << 30),
                                       B, H, F, T, d, masks, 0.125, None, None)
    with open(os.path.join(ROOT, "include", "tile_attn.h")) as f:
        hdr = f.read()
    assert "#define TA_NOALLOC_PLAN_WORDS 65536" in hdr
