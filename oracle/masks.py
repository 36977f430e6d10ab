"""Frame-tile masks of the k:(F-k) family and their block sparsity (oracle side).

Test infrastructure only; see the package docstring.

The paper keeps the tiles on the main diagonal and, off the diagonal, only the
attention against k "global reference frames" picked uniformly from the F
latent frames (Sec. 3.3 and the 2:6 example figure of Sec. 3.1). Two readings
of "attention against the reference frames" are provided:

* ``col``: query frame i keeps key frame i and every key frame in G.
* ``sym``: ``col`` plus every query frame in G keeps all key frames.

Placement of G: frames 0, s, 2s, ... below F with stride s = ceil(F / k).
Only the ``sym`` reading with this placement reproduces the sparsities printed
in tab:kernel_time (Sec. 4.2.1) when sparsity is counted over 128 x 128 blocks
of the flattened score matrix, and the same rule reproduces tab:cog_kernel
(App. E) under the stated CogVideoX shape assumptions.
"""
from __future__ import annotations

import math

import numpy as np

FORMS = ("col", "sym", "dense")


def global_frames(F: int, k: int) -> list[int]:
    """The k global reference frames, chosen uniformly from F frames (Sec. 3.3).

    Frames 0, s, 2s, ... below F with s = ceil(F / k); k = 0 gives none.
    """
    if F < 1 or k < 0 or k > F:
        raise ValueError(f"need F >= 1 and 0 <= k <= F, got F={F}, k={k}")
    if k == 0:
        return []
    stride = math.ceil(F / k)
    return list(range(0, F, stride))


def tile_mask(F: int, k: int, form: str = "col") -> np.ndarray:
    """F x F uint8 mask, row = query frame, column = key frame; 1 = tile kept."""
    if form not in FORMS:
        raise ValueError(f"form must be one of {FORMS}")
    M = np.zeros((F, F), dtype=np.uint8)
    if form == "dense":
        M[:, :] = 1
        return M
    G = global_frames(F, k)
    for i in range(F):
        M[i, i] = 1  # main diagonal tile
        for j in G:
            M[i, j] = 1  # attention against each global reference frame
    if form == "sym":
        for i in G:
            M[i, :] = 1  # the reference frames themselves attend to every frame
    return M


def nnz(mask: np.ndarray) -> int:
    """Number of kept tiles."""
    return int(np.count_nonzero(mask))


def tile_sparsity(mask: np.ndarray) -> float:
    """Fraction of frame tiles that are skipped."""
    return 1.0 - nnz(mask) / mask.size


def block_sparsity(mask: np.ndarray, T: int, block: int = 128, prefix: int = 0) -> float:
    """Fraction of block x block tiles of the score matrix that are entirely masked.

    This is the paper's "proportion of elements in the kernel that can be
    skipped" (Sec. 4.2.1) for a block-sparse kernel with 128 x 128 blocks over
    the flattened sequence; blocks straddle frame boundaries when T is not a
    multiple of the block size.

    ``prefix`` tokens (text tokens placed before the video in an MM-DiT,
    App. E) attend to everything and are attended by everything.
    """
    mask = np.asarray(mask).astype(bool)
    F = mask.shape[0]
    S = prefix + F * T
    nb = -(-S // block)
    # touches[b, f]: block b contains a token of frame f (f = F means the prefix)
    touches = np.zeros((nb, F + 1), dtype=bool)
    for b in range(nb):
        tok = np.arange(b * block, min(S, (b + 1) * block))
        frames = np.where(tok < prefix, F, (tok - prefix) // T)
        touches[b, np.unique(frames)] = True
    full = np.ones((F + 1, F + 1), dtype=bool)
    full[:F, :F] = mask
    t = touches.astype(np.int64)
    kept = (t @ full.astype(np.int64) @ t.T) > 0
    return 1.0 - kept.mean()
