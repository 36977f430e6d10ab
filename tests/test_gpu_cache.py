"""The bounded plan cache on the GPU: many distinct masks keep it at its capacity, and
a mask whose plan was evicted (and freed once its kernels finished) is planned again
and still matches the oracle."""
import numpy as np
import pytest

import workloads
from oracle import attention as oa
from tests.gpu_helpers import assert_parity, from_dev, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2502_06155_amd as ta  # noqa: E402

CAP = 256  # TA_PLAN_CACHE_ENTRIES


def test_many_masks_stay_within_the_cache_and_evicted_plans_still_work():
    B, H, F, T, d = 1, 2, 6, 40, 64
    qb, kb, vb = workloads.make_qkv(B, H, F, T, d, seed=140)
    q, k, v = (to_dev(x) for x in (qb, kb, vb))
    scale = d ** -0.5
    s = torch.cuda.current_stream()
    rng = np.random.default_rng(141)
    first = (rng.random((F, F)) < 0.5).astype(np.uint8)
    first[0, :] = 1  # a split heavy row: merge kernel and workspace too
    out0 = torch.empty_like(q)
    ta.tile_attn_fwd(q, k, v, out0, B, H, F, T, d, first, scale, s)
    torch.cuda.synchronize()
    ref0 = from_dev(out0)
    assert_parity(ref0, oa.attention(qb, kb, vb, first, T, scale), "cache-first")
    # 2^36 masks exist at F = 6: draw distinct ones, all different from `first`
    seen = {first.tobytes()}
    outs = []
    while len(seen) < 3 * CAP:
        m = (rng.random((F, F)) < 0.5).astype(np.uint8)
        if m.tobytes() in seen:
            continue
        seen.add(m.tobytes())
        o = torch.empty_like(q)
        ta.tile_attn_fwd(q, k, v, o, B, H, F, T, d, m, scale, s)  # queued without waits
        if len(outs) < 4 or len(seen) % 97 == 0:
            outs.append((m, o))
        live, retired = ta.tile_attn_plan_cache_stats()
        assert live <= CAP, live
    torch.cuda.synchronize()
    live, retired = ta.tile_attn_plan_cache_stats()
    print(f"[cache] live {live} retired {retired}", flush=True)
    assert live == CAP and retired == 0
    for m, o in outs:
        assert_parity(from_dev(o), oa.attention(qb, kb, vb, m, T, scale), "cache-evicting")
    # `first` was evicted long ago: planned and uploaded again, same result bit for bit
    out1 = torch.empty_like(q)
    ta.tile_attn_fwd(q, k, v, out1, B, H, F, T, d, first, scale, s)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(out1), ref0)
