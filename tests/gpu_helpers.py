"""Helpers shared by the GPU tests: moving bf16 bit patterns to and from the
device, and the parity gate against the float64 oracle."""
from __future__ import annotations

import numpy as np

# Parity gate for bf16 inputs with fp32 accumulation and bf16 output.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
# Diagnostic gate: an honest bf16 path sits near 2e-3; dropping frame-tail keys
# or using the wrong kept set lands far above it.
REL_RMS = 1e-2


def to_dev(bits: np.ndarray):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to("cuda", non_blocking=False)


def from_dev(t) -> np.ndarray:
    import torch

    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def widen(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def errors(got_bits: np.ndarray, ref: np.ndarray) -> dict:
    got = widen(got_bits)
    diff = np.abs(got - ref)
    rms_ref = float(np.sqrt(np.mean(ref * ref))) or 1.0
    return {
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "mean_abs": float(diff.mean()) if diff.size else 0.0,
        "rel_rms": float(np.sqrt(np.mean(diff * diff)) / rms_ref) if diff.size else 0.0,
        "finite": bool(np.all(np.isfinite(got))),
    }


def assert_parity(got_bits, ref, what=""):
    e = errors(got_bits, ref)
    print(f"[parity] {what} {e}", flush=True)
    assert e["finite"], f"{what}: non-finite output"
    assert e["max_abs"] <= MAX_ABS, f"{what}: max abs {e['max_abs']}"
    assert e["mean_abs"] <= MEAN_ABS, f"{what}: mean abs {e['mean_abs']}"
    assert e["rel_rms"] <= REL_RMS, f"{what}: rel rms {e['rel_rms']}"
    return e


def sample_rows(B, H, F, T, per_frame=4, heads=None, seed=0):
    """(b, h, s) rows to check at full size: first, last and ragged-tail rows of every
    frame plus random rows, for every (b, h) or the listed heads."""
    rng = np.random.default_rng(seed)
    bs, hs, ss = [], [], []
    tail = T - (T % 128) if T % 128 else T - 1
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            for f in range(F):
                rows = {0, T - 1, min(tail, T - 1), T // 2}
                rows |= set(int(x) for x in rng.integers(0, T, per_frame))
                for r in sorted(rows):
                    bs.append(b)
                    hs.append(h)
                    ss.append(f * T + r)
    return np.array(bs), np.array(hs), np.array(ss)


# Inputs of the named workloads, drawn once per process: the 93-frame shapes take tens
# of seconds of host time to draw and round, and several test modules use them.
_WORKLOAD_INPUTS = {}


def workload_inputs(name: str):
    """(qb, kb, vb) bf16 bits of workloads.WORKLOADS[name] (its own seed and recipe)."""
    import workloads

    if name not in _WORKLOAD_INPUTS:
        _WORKLOAD_INPUTS[name] = workloads.make_workload_qkv(workloads.WORKLOADS[name])
    return _WORKLOAD_INPUTS[name]


_GRADS = {}


def upstream_grad(shape, seed: int):
    """An N(0, 1) upstream gradient as bf16 bits from its own PCG64 stream, cached."""
    import workloads

    key = (tuple(shape), seed)
    if key not in _GRADS:
        rng = np.random.default_rng(seed)
        _GRADS[key] = workloads.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))
    return _GRADS[key]
