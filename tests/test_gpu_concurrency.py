"""Several host threads calling the library at once, each on its own stream: the
first calls for each thread's masks build their kept lists concurrently, and split
rows use per-stream workspaces. Every result must equal, bit for bit, the same call
made alone afterwards; those lone results are checked against the float64 oracle,
so a kept list corrupted while it was built would not go unnoticed."""
import threading

import numpy as np
import pytest

import workloads
from oracle import attention as oa
from oracle import backward as ob
from tests.gpu_helpers import assert_parity, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402

N_THREADS = 4
N_ITER = 5
# Same gate as the gradient parity tests: relative to each tensor's own scale.
GRAD_REL_RMS = 1e-2
GRAD_MAX_REL = 2e-2


def _case(i):
    B, H, F, T, d = 1, 3, 5 + i, 97 + 41 * i, (64, 96, 128, 96)[i]
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=300 + i)
    rng = np.random.default_rng(400 + i)
    gb = workloads.f32_to_bf16_bits(rng.standard_normal((B, H, F * T, d)).astype(np.float32))
    masks = (rng.random((H, F, F)) < 0.35).astype(np.uint8)
    masks[:, :, 0] = 1  # every query frame keeps frame 0: a heavy key column (split, summed)
    masks[0, 0, :] = 1  # one query frame keeps everything: a heavy row (split, merged)
    masks[1, 1, :] = 0  # and one keeps nothing
    return dict(B=B, H=H, F=F, T=T, d=d, scale=d ** -0.5, bits=(qb, kb, vb, gb), masks=masks)


def _device_case(c):
    q, k, v, g = (to_dev(x) for x in c["bits"])
    return q, k, v, g


def _outputs(q, n):
    S = q.shape[2]
    out = [torch.full_like(q, float("nan")) for _ in range(n)]
    lse = [torch.full((q.shape[0], q.shape[1], S), 12345.0, dtype=torch.float32, device="cuda")
           for _ in range(n)]
    grads = [[torch.full_like(q, float("nan")) for _ in range(3)] for _ in range(n)]
    return out, lse, grads


def _call(c, dev, out, lse, grads, stream):
    q, k, v, g = dev
    ta.tile_attn_fwd_heads(q, k, v, out, c["B"], c["H"], c["F"], c["T"], c["d"], c["masks"],
                           c["scale"], lse, stream)
    ta.tile_attn_bwd(q, k, v, out, g, lse, *grads, c["B"], c["H"], c["F"], c["T"], c["d"],
                     c["masks"], c["scale"], stream)


def _assert_grad(got_bits, ref, what):
    got = widen(got_bits)
    diff = np.abs(got - ref)
    peak = float(np.max(np.abs(ref)))
    rms = float(np.sqrt(np.mean(ref * ref)))
    print(f"[grad] {what} max_rel {diff.max() / peak:.2e} rel_rms "
          f"{np.sqrt(np.mean(diff * diff)) / rms:.2e}", flush=True)
    assert np.all(np.isfinite(got)), what
    assert diff.max() <= GRAD_MAX_REL * peak, what
    assert np.sqrt(np.mean(diff * diff)) <= GRAD_REL_RMS * rms, what


def test_threads_on_own_streams_match_lone_calls():
    cases = [_case(i) for i in range(N_THREADS)]
    devs = [_device_case(c) for c in cases]
    bufs = [_outputs(dv[0], N_ITER) for dv in devs]
    streams = [torch.cuda.Stream() for _ in range(N_THREADS)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())  # the inputs were copied on this one
    errors = []

    def worker(i):
        try:
            out, lse, grads = bufs[i]
            for it in range(N_ITER):
                _call(cases[i], devs[i], out[it], lse[it], grads[it], streams[i])
            streams[i].synchronize()
        except Exception as e:  # reported by the main thread
            errors.append((i, repr(e)))

    print(f"[case] {N_THREADS} threads x {N_ITER} forward+gradient calls", flush=True)
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(N_THREADS)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()

    for i, c in enumerate(cases):
        ro, rl, rg = _outputs(devs[i][0], 1)
        _call(c, devs[i], ro[0], rl[0], rg[0], torch.cuda.current_stream())
        torch.cuda.synchronize()
        ref_out, ref_lse = from_dev(ro[0]), rl[0].cpu().numpy()
        ref_grads = [from_dev(x) for x in rg[0]]
        out, lse, grads = bufs[i]
        for it in range(N_ITER):
            assert np.array_equal(from_dev(out[it]), ref_out), (i, it, "out")
            assert np.array_equal(lse[it].cpu().numpy(), ref_lse), (i, it, "lse")
            for name, a, r in zip(("dq", "dk", "dv"), grads[it], ref_grads):
                assert np.array_equal(from_dev(a), r), (i, it, name)
        qb, kb, vb, gb = c["bits"]
        assert_parity(ref_out, oa.attention(qb, kb, vb, c["masks"], c["T"], c["scale"]),
                      f"thread-case-{i}")
        refs = ob.attention_backward(qb, kb, vb, gb, c["masks"], c["T"], c["scale"])
        for name, a, r in zip(("dq", "dk", "dv"), ref_grads, refs):
            _assert_grad(a, r, f"thread-case-{i}-{name}")
