"""Benchmark of the tile-sparse attention forward on one MI355X.

One step = one tile_attn_fwd call (kept-tile list cached after the first call,
one kernel launch) over the 93-frame 720p-shaped problem: B=1, H=24, d=96,
F=24 latent frames x T=3600 tokens, mask = diagonal + 1 global frame (col
form), bf16 inputs resident in HBM. The mask is static (built once, outside the
timed region), as in the paper's kernel benchmark.

Prints ONE JSON line with the throughput over kept tiles, the roofline of the
attention kernel, the dense control and the CPU oracle baseline.

--pass bwd times the gradients instead: one step = one tile_attn_bwd call (prep,
dq pass, dk/dv pass, sums of split frames) on the same problem, with out and the
row log-sum-exp from one forward call made before the timed region. Its FLOP count
is the usual five products per kept tile (S = QK^T, dP = dO V^T, dV = P^T dO,
dK = dS^T Q, dQ = dS K): 10 * B * H * d * T^2 per kept tile.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

# MI355X dense bf16 matrix peak: 256 CUs x 4096 FLOP/clk x 2.4 GHz (the published 2.5 PFLOP/s).
PEAK_BF16_TFLOPS = 256 * 4096 * 2.4e9 / 1e12
CSRC = os.path.join(ROOT, "paper_2502_06155_amd", "csrc")
KERNEL_SRCS = {
    "fwd": [os.path.join(CSRC, f) for f in ("tile_attn_kernels.hip", "tile_common.h", "launch.h")],
    "bwd": [os.path.join(CSRC, f) for f in ("tile_attn_bwd.hip", "tile_common.h", "launch.h")],
}


def profile_md(which: str = "fwd", workload: str = "93f", form: str = "col", g: int = 1) -> str:
    """The committed rocprofv3 summary of one pass of one workload and mask:
    profiles/tile_attn_<pass>_<workload>_<form>_g<g>.md."""
    return os.path.join(ROOT, "profiles", f"tile_attn_{which}_{workload}_{form}_g{g}.md")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kept_flop(w, nnz: int, which: str = "fwd") -> float:
    """Forward: QK^T and PV over kept tiles only, 4 * B * H * d * T^2 per kept tile.
    Backward: the five products of the gradients, 10 * B * H * d * T^2 per kept tile.
    With a text prefix of P tokens (MM-DiT form) every query also attends the text and
    the text queries attend everything: 4 * B * H * d * (T^2 nnz + F T P + P S)."""
    per = 4.0 if which == "fwd" else 10.0
    pairs = float(w.T) ** 2 * nnz + float(w.prefix) * (w.F * w.T + w.S)
    return per * w.B * w.H * w.d * pairs


def time_calls(fn, steps: int, warmup: int, torch):
    """Warm up, then time exactly `steps` calls with events on the launch stream.

    Returns (total_ms, per_call_ms list)."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record(stream)
    for i in range(steps):
        fn()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return ev[0].elapsed_time(ev[-1]), per


def paper_stat(per_call):
    """Median and mean of the 20th-80th percentile band (the paper's protocol, Sec. 4.2.1)."""
    a = np.sort(np.asarray(per_call))
    lo, hi = np.percentile(a, 20), np.percentile(a, 80)
    band = a[(a >= lo) & (a <= hi)]
    return float(np.median(a)), float(band.mean() if band.size else a.mean())


def profile_record(which: str = "fwd", key: str = "hbm_bytes_per_launch", workload: str = "93f",
                   form: str = "col", g: int = 1):
    """One per-launch figure of the committed rocprofv3 counter summary of this pass,
    workload and mask, or None when there is none or it was taken on other kernel
    sources. hbm_bytes_per_launch: HBM bytes (FETCH_SIZE and WRITE_SIZE, each
    calibrated on a plain copy of known size); mfma_bf16_flop_per_launch:
    SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 FLOP per op."""
    path = profile_md(which, workload, form, g)
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("|", "#", " ", "`")):
                k, _, val = line.partition(":")
                rec[k.strip()] = val.strip()
    sha = hashlib.sha256(b"".join(open(p, "rb").read() for p in KERNEL_SRCS[which])).hexdigest()
    if rec.get("kernel_sha256") != sha or key not in rec:
        return None
    return float(rec[key])


def traffic_from_profile(which: str = "fwd", workload: str = "93f", form: str = "col", g: int = 1):
    """HBM bytes per launch of the dominant kernel(s), or None (see profile_record)."""
    return profile_record(which, "hbm_bytes_per_launch", workload, form, g)


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), for the baseline's record."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(w, qb, kb, vb, mask, budget_s: float):
    """Time the float64 oracle on whole heads of the same problem until the budget
    is spent; report kept TFLOP/s of that sample."""
    from oracle import attention as oa

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    from oracle import mmdit as ommd

    nnz = int(np.count_nonzero(mask))
    done, t0 = 0, time.perf_counter()
    while done < w.H and time.perf_counter() - t0 < budget_s:
        sl = slice(done, done + 1)
        if w.prefix:
            ommd.attention_mmdit(qb[:, sl], kb[:, sl], vb[:, sl], mask, w.T, w.prefix, w.scale())
        else:
            oa.attention(qb[:, sl], kb[:, sl], vb[:, sl], mask, w.T, w.scale())
        done += 1
    dt = time.perf_counter() - t0
    flop = kept_flop(w, nnz) * done / w.H
    return {
        "value": flop / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"float64 numpy oracle (the parity reference, kept in float64 so its rounding "
                  f"is negligible next to bf16) on heads 0..{done - 1} of {w.H} (all {w.F} query "
                  f"frames, b=0) of the same problem, {dt:.1f} s; throughput over kept tiles; "
                  f"{cpu_model()}",
    }


def cpu_baseline_bwd(w, qb, kb, vb, gb, mask, budget_s: float):
    """The float64 gradient oracle on whole heads of the same problem until the budget
    is spent; kept TFLOP/s of that sample (five products per kept tile)."""
    from oracle import backward as ob

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    nnz = int(np.count_nonzero(mask))
    done, t0 = 0, time.perf_counter()
    from oracle import mmdit as ommd

    while done < w.H and time.perf_counter() - t0 < budget_s:
        sl = slice(done, done + 1)
        if w.prefix:
            ommd.attention_backward_mmdit(qb[:, sl], kb[:, sl], vb[:, sl], gb[:, sl], mask, w.T, w.prefix,
                                          w.scale())
        else:
            ob.attention_backward(qb[:, sl], kb[:, sl], vb[:, sl], gb[:, sl], mask, w.T, w.scale())
        done += 1
    dt = time.perf_counter() - t0
    flop = kept_flop(w, nnz, "bwd") * done / w.H
    return {
        "value": flop / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"float64 numpy gradient oracle (the parity reference) on heads 0..{done - 1} of "
                  f"{w.H} (all {w.F} frames, b=0) of the same problem, {dt:.1f} s; throughput over "
                  f"kept tiles; {cpu_model()}",
    }


def make_grad_bits(w, seed: int = 1):
    """Upstream gradient dO: N(0, 1) per element as bf16 bits, one PCG64 stream."""
    rng = np.random.default_rng(seed)
    return workloads.f32_to_bf16_bits(
        rng.standard_normal((w.B, w.H, w.S, w.d), dtype=np.float32))


class Problem:
    """Device tensors of one workload and a step closure for one mask and pass."""

    def __init__(self, torch, ta, w, qb, kb, vb, which: str):
        self.torch, self.ta, self.w, self.which = torch, ta, w, which

        def dev(x):
            return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()

        self.q, self.k, self.v = dev(qb), dev(kb), dev(vb)
        self.out = torch.empty_like(self.q)
        if which == "bwd":
            self.gb = make_grad_bits(w)
            self.dout = dev(self.gb)
            self.lse = torch.empty((w.B, w.H, w.S), dtype=torch.float32, device="cuda")
            self.grads = [torch.empty_like(self.q) for _ in range(3)]
        self.stream = torch.cuda.current_stream()

    def step_fn(self, mask):
        w, ta, st = self.w, self.ta, self.stream
        q, k, v, out = self.q, self.k, self.v, self.out
        if self.which == "fwd" and w.prefix:
            return lambda: ta.tile_attn_fwd_mmdit(q, k, v, out, w.B, w.H, w.F, w.T, w.prefix, w.d, mask,
                                                  w.scale(), None, st)
        if self.which == "fwd":
            return lambda: ta.tile_attn_fwd(q, k, v, out, w.B, w.H, w.F, w.T, w.d, mask, w.scale(), st)
        # out and lse of this mask, once, outside the timed region
        dq, dk, dv = self.grads
        if w.prefix:
            ta.tile_attn_fwd_mmdit(q, k, v, out, w.B, w.H, w.F, w.T, w.prefix, w.d, mask, w.scale(),
                                   self.lse, st)
            return lambda: ta.tile_attn_bwd_mmdit(q, k, v, out, self.dout, self.lse, dq, dk, dv, w.B,
                                                  w.H, w.F, w.T, w.prefix, w.d, mask, w.scale(), st)
        ta.tile_attn_fwd_heads(q, k, v, out, w.B, w.H, w.F, w.T, w.d, mask, w.scale(), self.lse, st)
        return lambda: ta.tile_attn_bwd(q, k, v, out, self.dout, self.lse, dq, dk, dv, w.B, w.H, w.F,
                                        w.T, w.d, mask, w.scale(), st)


def gemm_reference(torch, n: int = 16384, reps: int = 5):
    """Dense bf16 GEMM (torch.matmul, i.e. the vendor BLAS) on N(0,1) data of the same
    GPU: the matrix-core rate this chip sustains on random data under its power
    limit, reported beside the published peak as context."""
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    for _ in range(2):
        a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return {"shape": f"{n}x{n}x{n} bf16 N(0,1), torch.matmul", "ms": ms,
            "tflops": 2.0 * n ** 3 / (ms * 1e-3) / 1e12}


# Every workload of the measurement plan: (workload, mask form, g). The dense control is
# timed once per workload.
ALL_CASES = [
    ("tiny", "col", 1), ("tiny", "sym", 1),
    ("29f", "col", 1), ("29f", "sym", 1),
    ("93f", "col", 1), ("93f", "sym", 1),
    ("sweep", "col", 1), ("sweep", "col", 2), ("sweep", "col", 4), ("sweep", "col", 8),
    ("sweep", "sym", 2), ("sweep", "sym", 4), ("sweep", "sym", 8),
    ("sp_share", "col", 1), ("sp_share", "sym", 1),
    ("long", "col", 2), ("long", "sym", 2),
    ("93f_d128", "col", 1), ("93f_d128", "sym", 1),
    # MM-DiT form at the CogVideoX-5B shape: tab:cog_kernel labels 12, 6, 4, 3, 2, 1 are
    # k = 1, 2, 3, 4, 6, 12 global frames (sym form).
    ("cog", "sym", 1), ("cog", "sym", 2), ("cog", "sym", 3), ("cog", "sym", 4),
    ("cog", "sym", 6), ("cog", "sym", 12),
]


def run_all(args, torch, ta):
    """Time every case of ALL_CASES and the dense control of each workload; print one
    table row per case to stderr and return the rows."""
    rows, cur, dense_ms = [], None, {}
    order = []
    for wname in dict.fromkeys(c[0] for c in ALL_CASES):
        order += [c for c in ALL_CASES if c[0] == wname] + [(wname, "dense", 0)]
    for name, form, g in order:
        w = workloads.WORKLOADS[name]
        if cur is None or cur.w.name != name:
            cur = None
            qb, kb, vb = workloads.make_workload_qkv(w)
            cur = Problem(torch, ta, w, qb, kb, vb, args.pass_)
            del qb, kb, vb
        mask = ta.tile_attn_make_mask(w.F, g, form)
        nnz = int(np.count_nonzero(mask))
        step = cur.step_fn(mask)
        steps = max(3, min(args.steps, int(2000 / max(1.0, nnz))))
        # Keep the GPU busy for about half a second first: after the host-side input
        # generation of a new workload the clocks have dropped, which a fixed count of
        # warm-up calls on a short case does not undo.
        t0, n = time.perf_counter(), 0
        while n < 2 or time.perf_counter() - t0 < 0.5:
            step()
            torch.cuda.synchronize()
            n += 1
        total, per = time_calls(step, steps, 0, torch)
        ms = total / steps
        tf = kept_flop(w, nnz, args.pass_) / (ms * 1e-3) / 1e12
        if form == "dense":
            dense_ms[name] = ms
        row = {"workload": name, "form": form, "g": g, "nnz": nnz, "tiles": w.F * w.F, "ms": ms,
               "tflops": tf, "pct_peak": 100.0 * tf / PEAK_BF16_TFLOPS}
        rows.append(row)
        log(f"[all] {args.pass_} {name:8s} {form:5s} g={g} nnz {nnz:4d}/{w.F * w.F:<4d} {ms:9.3f} ms "
            f"{tf:7.1f} TFLOP/s ({row['pct_peak']:.1f}% of peak)")
    for row in rows:
        if row["workload"] in dense_ms and row["form"] != "dense":
            row["speedup_vs_dense"] = dense_ms[row["workload"]] / row["ms"]
            row["ideal_speedup"] = row["tiles"] / row["nnz"]
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the paper's protocol (Sec. 4.2.1): 25 warm-up calls, then 100 timed ones
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default="93f", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--form", default="col", choices=["col", "sym", "dense"])
    ap.add_argument("--g", type=int, default=None)
    ap.add_argument("--pass", dest="pass_", default="fwd", choices=["fwd", "bwd"],
                    help="fwd: the attention forward (headline); bwd: its gradients")
    ap.add_argument("--dense-steps", type=int, default=5)
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-gemm-ref", action="store_true")
    ap.add_argument("--profile-pass", action="store_true",
                    help="counter pass: sparse calls, then a plain copy of --copy-mib MiB "
                         "(the calibration kernel for HBM byte counters); no dense, no CPU")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--all", action="store_true",
                    help="time every workload and mask of the measurement plan instead of the "
                         "headline; prints one JSON line with a row per case")
    args = ap.parse_args()
    if args.profile_pass:
        args.no_dense = True
        args.no_cpu_baseline = True
        args.no_gemm_ref = True

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the attention "
              "shards over heads with no exchange inside the op, so N GPUs each run this "
              "kernel on H/N heads.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2502_06155_amd as ta

    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)

    if args.all:
        rows = run_all(args, torch, ta)
        print(json.dumps({"metric": f"per-case ms/call and TFLOP/s over kept tiles ({args.pass_})",
                          "unit": "TFLOP/s",
                          "n_gpus": 1, "dtype": "bf16", "data": "synthetic", "rows": rows}), flush=True)
        return

    w = workloads.WORKLOADS[args.workload]
    g = w.g if args.g is None else args.g
    which = args.pass_
    log(f"[bench] workload {w} form={args.form} g={g} pass={which}")
    qb, kb, vb = workloads.make_workload_qkv(w)
    mask = ta.tile_attn_make_mask(w.F, g, args.form)
    nnz = int(np.count_nonzero(mask))
    prob = Problem(torch, ta, w, qb, kb, vb, which)
    step = prob.step_fn(mask)

    torch.cuda.synchronize()
    total_ms, per = time_calls(step, args.steps, args.warmup, torch)
    ms = total_ms / args.steps
    med, band = paper_stat(per)
    flop = kept_flop(w, nnz, which)
    tflops = flop / (ms * 1e-3) / 1e12
    log(f"[bench] sparse {which}: {ms:.3f} ms/call (median {med:.3f}, P20-P80 {band:.3f}), "
        f"{tflops:.1f} TFLOP/s kept, nnz {nnz}/{w.F * w.F}")

    if args.profile_pass:
        # A plain elementwise copy that reads and writes exactly copy_mib MiB each: the
        # same HBM counters read on it give the factor from counter units to bytes.
        n = args.copy_mib * (1 << 20) // 2
        src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: 3 x torch.neg over {args.copy_mib} MiB in, {args.copy_mib} MiB out")

    extra = {}
    if not args.no_dense:
        dstep = prob.step_fn(np.ones((w.F, w.F), np.uint8))
        dtot, dper = time_calls(dstep, args.dense_steps, 2, torch)
        dms = dtot / args.dense_steps
        dflop = kept_flop(w, w.F * w.F, which)
        extra = {
            "dense_ms_per_call": dms,
            "dense_tflops": dflop / (dms * 1e-3) / 1e12,
            "speedup_vs_dense": dms / ms,
            "ideal_speedup": w.F * w.F / nnz,
        }
        extra["proportionality"] = tflops / extra["dense_tflops"]
        log(f"[bench] dense {which}: {dms:.3f} ms/call, {extra['dense_tflops']:.1f} TFLOP/s, "
            f"speedup {extra['speedup_vs_dense']:.2f}x of ideal {extra['ideal_speedup']:.2f}x")

    gemm = None
    if not args.no_gemm_ref:
        gemm = gemm_reference(torch)
        log(f"[bench] vendor bf16 GEMM on random data: {gemm['tflops']:.1f} TFLOP/s")

    cpu = None
    if not args.no_cpu_baseline:
        if which == "fwd":
            cpu = cpu_baseline(w, qb, kb, vb, mask, args.cpu_budget)
        else:
            cpu = cpu_baseline_bwd(w, qb, kb, vb, prob.gb, mask, args.cpu_budget)
        log(f"[bench] cpu oracle: {cpu}")

    achieved = flop / (np.mean(per) * 1e-3) / 1e12
    metric = "ms/call + effective TFLOP/s (kept tiles) and % bf16 MFMA peak, 24f×3600 tok"
    if which == "bwd":
        metric = ("backward ms/call + effective TFLOP/s (kept tiles, five products) and % bf16 "
                  "MFMA peak, 24f×3600 tok")
    line = {
        "metric": metric,
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_median": med,
        "ms_p20_p80_mean": band,
        "pct_bf16_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: B={w.B} H={w.H} F={w.F} T={w.T} d={w.d}, "
                        f"{args.form} mask g={g} (nnz {nnz}/{w.F * w.F}), {w.dist} N(0,1) bf16 seed {w.seed}",
            "pass": which,
            "kept_flop": flop,
            "nnz": nnz,
        },
        "roofline": {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic_from_profile(which, w.name, args.form, g),
        },
        "cpu_baseline": cpu,
        "gemm_reference": gemm,
    }
    # Matrix work the counters saw (padding included) over the same measured time.
    mfma_flop = profile_record(which, "mfma_bf16_flop_per_launch", w.name, args.form, g)
    if mfma_flop is not None:
        ctf = mfma_flop / (np.mean(per) * 1e-3) / 1e12
        line["mfma_counter"] = {"flop_per_launch": mfma_flop, "tflops": ctf,
                                "frac": ctf / PEAK_BF16_TFLOPS,
                                "source": "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512, "
                                          + os.path.relpath(profile_md(which, w.name, args.form, g), ROOT)}
    line.update(extra)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
