"""The one-call Python entry points (dedup, merge_retrieval) against the
oracle: canonical dedup bit-exact, every request's result accepted against
an independent retrieval of its own query row (Sec. 3.3 (I): the merged
result equals each request's own retrieval), workflow slices."""
import numpy as np
import pytest
import torch

import synth
from gpu_harness import check_requests_vs_oracle, check_unique_topk, device, to_dev

pytestmark = pytest.mark.gpu


def test_dedup_one_call():
    import oracle
    import paper_2607_22578_amd as hs
    rng = np.random.default_rng(3)
    for R in (0, 1, 1000, 5000, 70_000):
        keys = rng.integers(-50, 50, size=R).astype(np.int64) * (1 << 40)
        uk, fi, ct, inv = hs.dedup(torch.from_numpy(keys).to(device()))
        ref = oracle.dedup(keys)
        assert uk.shape[0] == ref["n_unique"]
        np.testing.assert_array_equal(uk.cpu().numpy(), ref["unique_keys"])
        np.testing.assert_array_equal(fi.cpu().numpy(), ref["first_index"])
        np.testing.assert_array_equal(ct.cpu().numpy(), ref["counts"])
        np.testing.assert_array_equal(inv.cpu().numpy(), ref["inverse"])


@pytest.mark.parametrize("enc", ["bf16", "fp8"])
def test_merge_retrieval_one_call(enc):
    import paper_2607_22578_amd as hs
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    N = 12_000
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, N, w.dim, enc)
    # uneven workflows over the window's requests
    offs = np.concatenate([[0], np.sort(np.random.default_rng(5).choice(
        np.arange(1, w.R), size=9, replace=False)), [w.R]])
    res = hs.merge_retrieval(to_dev(w.keys), to_dev(w.q_req), to_dev(c), w.k,
                             scale=to_dev(sc) if sc is not None else None,
                             workflow_offsets=offs)
    import oracle
    ref = oracle.dedup(w.keys)
    assert res["n_unique"] == ref["n_unique"]
    np.testing.assert_array_equal(res["unique_keys"].cpu().numpy(), ref["unique_keys"])
    np.testing.assert_array_equal(res["inverse"].cpu().numpy(), ref["inverse"])
    m = res["retrieval"]
    check_unique_topk(m, ref, w.q_req, c, w.k, scale=sc,
                      sel=np.array([0, 1, ref["n_unique"] // 2, ref["n_unique"] - 1]))
    reqs = np.array([0, 5, w.R // 3, w.R - 1])
    check_requests_vs_oracle(m, ref, reqs, w.q_req, c, w.k, scale=sc)
    # workflow w's rows are [offs[w], offs[w+1]) of the per-request outputs
    for wf in (0, 4, 9):
        s, i = m.workflow_results(wf)
        assert s.shape[0] == offs[wf + 1] - offs[wf]
        np.testing.assert_array_equal(i.cpu().numpy(),
                                      res["out_index"][offs[wf]:offs[wf + 1]].cpu().numpy())
