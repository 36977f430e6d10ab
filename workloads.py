"""Seeded synthetic inputs for tile-sparse 3D attention.

Shared by the tests, the benchmark and the smoke check. This module only draws
random numbers and rounds them to bf16; it holds none of the attention
arithmetic and none of the mask logic, so the GPU path and the CPU oracle stay
independent of each other.

Shapes follow the paper's 720p workloads (Sec. 4.1): the VAE compresses 8x in
space and the patch embedding another 2x, so a 720p latent frame is a 45 x 80
grid of T = 3600 tokens; 29 and 93 input frames give F = 8 and F = 24 latent
frames. Tokens are flattened frame-major (frame, then height, then width), so
token s belongs to latent frame s // T. The activations themselves are
synthetic stand-ins for Open-Sora-Plan attention inputs, which are not available.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    """One attention problem: [B, H, prefix + F*T, d] bf16 tensors plus a mask recipe
    (prefix = text tokens before the video in the MM-DiT form, else 0)."""

    name: str
    B: int
    H: int
    F: int
    T: int
    d: int
    g: int  # number of global reference frames in the k:(F-k) mask
    dist: str = "iid"  # "iid" or "frame_shift"
    seed: int = 0
    prefix: int = 0

    @property
    def S(self) -> int:
        return self.prefix + self.F * self.T

    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))


# The five workload families the build is measured and checked on.
WORKLOADS = {
    # 8 x 8 latent grid, 4 frames: small enough for exhaustive CPU checks.
    "tiny": Workload("tiny", B=1, H=2, F=4, T=64, d=64, g=1),
    # 29-frame 720p: 8 latent frames of 45 x 80 tokens.
    "29f": Workload("29f", B=1, H=24, F=8, T=3600, d=96, g=1),
    # 93-frame 720p: 24 latent frames of 45 x 80 tokens (headline shape).
    "93f": Workload("93f", B=1, H=24, F=24, T=3600, d=96, g=1),
    # Sparsity sweep at 93f with frame-correlated tokens; g is varied by callers.
    "sweep": Workload("sweep", B=1, H=24, F=24, T=3600, d=96, g=1, dist="frame_shift"),
    # One GPU's share of a 4-way head split of the 93f problem.
    "sp_share": Workload("sp_share", B=1, H=6, F=24, T=3600, d=96, g=1),
    # Long horizon: 48 latent frames of a 30 x 40 grid.
    "long": Workload("long", B=1, H=24, F=48, T=1200, d=96, g=2),
    # The 93-frame shape with 128-wide heads (18 heads keep the model width of 24 x 96).
    "93f_d128": Workload("93f_d128", B=1, H=18, F=24, T=3600, d=128, g=1),
    # MM-DiT form at the CogVideoX-5B shape of App. E: 49 frames -> 13 latent frames,
    # 480p -> 30 x 45 = 1350 tokens per frame, 226 text tokens first, 48 heads of 64.
    "cog": Workload("cog", B=1, H=48, F=13, T=1350, d=64, g=1, prefix=226),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bf16 (round to nearest, ties to even).

    Returns the bf16 bit patterns as uint16. Works through the array in pieces of
    2^20 values, which keeps the temporaries in cache for the large workloads.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    flat = x.reshape(-1)
    u = flat.view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    step = 1 << 20
    for i in range(0, u.size, step):
        if not np.all(np.isfinite(flat[i:i + step])):
            raise ValueError("only finite values are converted")
        c = u[i:i + step]
        r = (c >> np.uint32(16)) & np.uint32(1)
        r += np.uint32(0x7FFF)
        r += c
        r >>= np.uint32(16)
        out[i:i + step] = r
    return out.reshape(x.shape)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def make_qkv(B: int, H: int, F: int, T: int, d: int, seed: int = 0, dist: str = "iid",
             prefix: int = 0):
    """Draw Q, K, V as bf16 bit patterns of shape [B, H, prefix + F*T, d].

    iid: every element is N(0, 1).
    frame_shift: x = z + 0.5 * mu, with z ~ N(0, 1) per element and one
    mu ~ N(0, I_d) per (tensor, b, h, frame), so tokens of one frame share a
    mean, which mimics frame-correlated video tokens.

    One numpy PCG64 stream seeded with ``seed`` draws Q, K, V in that order,
    then (frame_shift only) the shifts for Q, K, V in that order. Text tokens
    (the first ``prefix``) are iid N(0, 1) and get no frame shift.
    """
    rng = np.random.default_rng(seed)
    S = prefix + F * T
    outs = []
    for _ in range(3):
        outs.append(rng.standard_normal((B, H, S, d), dtype=np.float32))
    if dist == "frame_shift":
        for x in outs:
            mu = rng.standard_normal((B, H, F, 1, d), dtype=np.float32)
            x[:, :, prefix:].reshape(B, H, F, T, d)[...] += np.float32(0.5) * mu
    elif dist != "iid":
        raise ValueError(f"unknown distribution {dist!r}")
    return tuple(f32_to_bf16_bits(x) for x in outs)


def make_workload_qkv(w: Workload):
    return make_qkv(w.B, w.H, w.F, w.T, w.d, seed=w.seed, dist=w.dist, prefix=w.prefix)
