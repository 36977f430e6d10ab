"""Pins of the oracle's mask family against the paper's printed sparsities (CPU only)."""
import math

import numpy as np
import pytest

from oracle import masks as om


def test_kernel_time_sparsities_reproduce_exactly(golden):
    """tab:kernel_time (Sec. 4.2.1): the sym reading with G = range(0, F, ceil(F/k)),
    counted over 128 x 128 blocks, gives every printed sparsity to two decimals."""
    for F, T, k, pct in golden("kernel_time_sparsity.txt"):
        F, T, k = int(F), int(T), int(k)
        sp = om.block_sparsity(om.tile_mask(F, k, "sym"), T)
        assert f"{100 * sp:.2f}" == pct, (F, k, 100 * sp, pct)


def test_col_reading_does_not_reproduce_kernel_time(golden):
    """The column-only reading is not what the paper timed."""
    mismatches = 0
    for F, T, k, pct in golden("kernel_time_sparsity.txt"):
        sp = om.block_sparsity(om.tile_mask(int(F), int(k), "col"), int(T))
        mismatches += f"{100 * sp:.2f}" != pct
    assert mismatches == 9


def test_other_placement_does_not_reproduce_3_5():
    """floor(i*F/k) placement gives {0, 2, 5} at F=8, k=3, which misses the printed 29.88."""
    F, k, T = 8, 3, 3600
    M = np.zeros((F, F), np.uint8)
    G = [i * F // k for i in range(k)]
    assert G == [0, 2, 5]
    for i in range(F):
        M[i, i] = 1
        M[i, G] = 1
    M[G, :] = 1
    assert f"{100 * om.block_sparsity(M, T):.2f}" != "29.88"
    assert om.global_frames(F, k) == [0, 3, 6]


def test_cog_kernel_sparsities_reproduce(golden):
    """tab:cog_kernel (App. E) under the stated CogVideoX shape reading."""
    for label, F, T, prefix, k, pct in golden("cog_kernel_sparsity.txt"):
        sp = om.block_sparsity(om.tile_mask(int(F), int(k), "sym"), int(T), prefix=int(prefix))
        assert f"{100 * sp:.2f}" == pct, (label, 100 * sp, pct)


@pytest.mark.parametrize("F", list(range(1, 49)))
def test_nnz_closed_forms(F):
    for k in range(0, F + 1):
        G = om.global_frames(F, k)
        g = len(G)
        assert g <= k and (k == 0 or G[0] == 0)
        assert om.nnz(om.tile_mask(F, k, "col")) == F * (g + 1) - g
        assert om.nnz(om.tile_mask(F, k, "sym")) == 2 * F * g + F - g * g - g
        assert om.nnz(om.tile_mask(F, k, "dense")) == F * F


def test_structure():
    for F, k in [(8, 2), (24, 4), (48, 2), (13, 6)]:
        col, sym = om.tile_mask(F, k, "col"), om.tile_mask(F, k, "sym")
        assert np.all(np.diag(col) == 1) and np.all(np.diag(sym) == 1)
        assert np.array_equal(sym, sym.T)
        assert np.all(sym >= col)
        G = om.global_frames(F, k)
        assert np.all(col[:, G] == 1) and np.all(sym[G, :] == 1)


def test_configured_global_frames():
    """Global frames of the measured workloads: G has exactly g frames in each."""
    assert om.global_frames(4, 1) == [0]
    assert om.global_frames(24, 1) == [0]
    assert om.global_frames(24, 2) == [0, 12]
    assert om.global_frames(24, 4) == [0, 6, 12, 18]
    assert om.global_frames(24, 8) == list(range(0, 24, 3))
    assert om.global_frames(48, 2) == [0, 24]
    assert om.global_frames(8, 1) == [0]


def test_tile_sparsity_linear_in_frames():
    """Constant kept tiles per row: nnz grows linearly in F (Sec. 3.3)."""
    for k in (1, 2, 4):
        counts = [om.nnz(om.tile_mask(F, k, "col")) for F in range(8, 65, 8)]
        diffs = np.diff(counts)
        assert np.all(diffs == diffs[0])


def test_block_sparsity_brute_force_small():
    """Block counting checked against an explicit token-level mask on small shapes."""
    rng = np.random.default_rng(0)
    for F, T, blk, prefix in [(3, 5, 4, 0), (4, 7, 8, 3), (2, 16, 16, 0), (5, 3, 4, 2)]:
        M = (rng.random((F, F)) < 0.4).astype(np.uint8)
        S = prefix + F * T
        frame = np.where(np.arange(S) < prefix, -1, (np.arange(S) - prefix) // T)
        tok = np.ones((S, S), bool)
        for a in range(S):
            for b in range(S):
                if frame[a] >= 0 and frame[b] >= 0:
                    tok[a, b] = bool(M[frame[a], frame[b]])
        nb = math.ceil(S / blk)
        skipped = 0
        for bi in range(nb):
            for bj in range(nb):
                skipped += not tok[bi * blk:(bi + 1) * blk, bj * blk:(bj + 1) * blk].any()
        assert om.block_sparsity(M, T, blk, prefix) == pytest.approx(skipped / nb ** 2, abs=1e-15)
