"""tile_attn_fwd_heads_noalloc (the forward that allocates no device memory: plan and
partials in the library's static per-GPU scratch array) against the existing entry
point tile_attn_fwd_heads and the oracle, on two calls in a row, the second smaller
(the scratch keeps the first call's contents)."""
import numpy as np
import pytest

import workloads
from oracle import attention as oa
from oracle import masks as om
from tests.gpu_helpers import assert_parity, from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402


def _both(qb, kb, vb, masks, T, scale):
    B, H, S, d = qb.shape
    F = S // T
    q, k, v = (to_dev(x) for x in (qb, kb, vb))
    s = torch.cuda.current_stream()
    out_a = torch.full_like(q, float("nan"))
    out_b = torch.full_like(q, float("nan"))
    lse_a = torch.full((B, H, S), float("nan"), dtype=torch.float32, device="cuda")
    lse_b = torch.full((B, H, S), float("nan"), dtype=torch.float32, device="cuda")
    ta.tile_attn_fwd_heads_noalloc(q, k, v, out_a, B, H, F, T, d, masks, scale, lse_a, s)
    ta.tile_attn_fwd_heads(q, k, v, out_b, B, H, F, T, d, masks, scale, lse_b, s)
    torch.cuda.synchronize()
    return from_dev(out_a), from_dev(out_b), lse_a.cpu().numpy(), lse_b.cpu().numpy()


def test_noalloc_matches_the_allocating_entry_point_on_two_calls():
    # call 1: split heavy query frames (the sym mask's global row), partials in scratch
    B, H, F, T, d = 2, 4, 10, 300, 96
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=150, dist="frame_shift")
    mask = om.tile_mask(F, 1, "sym")
    assert ta.tile_attn_plan(mask)[1] > 0
    print(f"[case] noalloc call 1 B={B} H={H} F={F} T={T} d={d} sym", flush=True)
    a, b, la, lb = _both(qb, kb, vb, mask, T, d ** -0.5)
    assert np.array_equal(a, b)
    assert np.array_equal(la, lb)
    assert_parity(a, oa.attention(qb, kb, vb, mask, T, d ** -0.5), "noalloc-1")
    # call 2, smaller: per-head masks with split rows and an empty query frame, d = 64
    B, H, F, T, d = 1, 2, 6, 100, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=151)
    masks = np.stack([om.tile_mask(F, 1, "sym"), om.tile_mask(F, 2, "col")])
    masks[1, 3, :] = 0
    print(f"[case] noalloc call 2 B={B} H={H} F={F} T={T} d={d} per-head", flush=True)
    a, b, la, lb = _both(qb, kb, vb, masks, T, 0.2)
    assert np.array_equal(a, b)
    assert np.array_equal(la, lb)
    assert_parity(a, oa.attention(qb, kb, vb, masks, T, 0.2), "noalloc-2")
    assert not np.any(a[0, 1, 3 * T:4 * T])
