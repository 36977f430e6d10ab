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
