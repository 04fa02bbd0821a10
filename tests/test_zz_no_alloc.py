"""The allocation-free score entry point (hs_score_topk_noalloc) against the
workspace one (hs_score_topk), through the C ABI: two calls in a row on one
GPU, the second with fewer distinct queries and a smaller corpus, each
bit-identical to the workspace entry point's results and accepted by the
oracle for a sample of queries; plans beyond the scratch size are rejected
before any launch."""
import numpy as np
import pytest
import torch

import synth
from gpu_harness import check_unique_topk, device, note, to_dev

pytestmark = pytest.mark.gpu


def _case(nu, N, seed):
    d, k = 768, 10
    q, _ = synth.gaussian_rows(seed, 31, nu, d, "bf16")
    c, _ = synth.gaussian_rows(seed, 32, N, d, "bf16")
    c[N // 3] = c[7]          # a planted exact tie
    return q, c, d, k


def _run(hs, q, c, d, k, nu, N, noalloc, plan):
    dev = device()
    qd, cd = to_dev(q), to_dev(c)
    ts = torch.full((nu, k), float("nan"), dtype=torch.float32, device=dev)
    ti = torch.full((nu, k), -7, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream(dev)
    if noalloc:
        hs.hs_score_topk_noalloc(plan, qd, nu, None, cd, None, ts, ti, stream=st)
    else:
        ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=dev)
        hs.hs_score_topk(plan, qd, nu, None, cd, None, ts, ti, ws, stream=st)
    torch.cuda.synchronize(dev)
    return ts.cpu().numpy(), ti.cpu().numpy()


def test_noalloc_matches_workspace_entry_point_twice():
    import paper_2607_22578_amd as hs
    for nu, N, seed in [(300, 120_000, 1), (45, 20_000, 2)]:
        q, c, d, k = _case(nu, N, seed)
        plan = hs.hs_merge_plan(nu, d, N, k, hs.HS_BF16, hs.HS_BF16)
        note(f"noalloc: n_u={nu} N={N} ws={plan.workspace_bytes}")
        s0, i0 = _run(hs, q, c, d, k, nu, N, False, plan)
        s1, i1 = _run(hs, q, c, d, k, nu, N, True, plan)
        np.testing.assert_array_equal(i1, i0)
        np.testing.assert_array_equal(s1.view(np.uint32), s0.view(np.uint32))

        class _M:   # the harness reads topk_* from an object
            pass
        m = _M()
        m.topk_score, m.topk_index = torch.from_numpy(s1), torch.from_numpy(i1)
        ref = {"n_unique": nu, "first_index": np.arange(nu, dtype=np.int32)}
        check_unique_topk(m, ref, q, c, k, sel=np.array([0, 7, nu // 2, nu - 1]))


def test_noalloc_rejects_plans_beyond_the_scratch():
    import paper_2607_22578_amd as hs
    big = hs.hs_merge_plan(32768, 1024, 4_000_000, 32, hs.HS_BF16, hs.HS_BF16)
    assert big.workspace_bytes > 64 << 20
    with pytest.raises(hs.HsError) as e:
        hs.hs_score_topk_noalloc(big, 0x10000000, 10, None, 0x10000000, None, 0x10000000,
                                 0x10000000)
    assert e.value.status == hs.HS_ERR_WORKSPACE
    assert "scratch" in hs.hs_last_error()
