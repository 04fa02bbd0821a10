"""Micro-batching of the distinct queries (Eq. 8's batching window and
split; Appendix A's batch limit B_r) leaves every result unchanged: scoring
the 1M-row workload's distinct queries in sequential sub-batches of at most
B queries, or as k sub-batches on k streams, gives top-k rows bit-identical
to one batch (each query's scores and its top-k do not depend on the other
queries of its batch), and one batch passes the acceptance rule against the
oracle."""
import numpy as np
import pytest
import torch

import synth
from gpu_harness import check_dedup, check_unique_topk, device, note, to_dev

pytestmark = pytest.mark.gpu


def _setup(n_corpus=20_000, enc="bf16", tiled=False):
    import paper_2607_22578_amd as hs
    dev = device()
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, w.dim, enc)
    m = hs.MergedRetrieval(w.R, w.dim, n_corpus, w.k, hs.HS_BF16,
                           hs.HS_BF16 if enc == "bf16" else hs.HS_FP8_E4M3, device=dev,
                           tiled_corpus=tiled)
    st = torch.cuda.current_stream(dev)
    kd, qd = to_dev(w.keys), to_dev(w.q_req)
    nu = m.dedup(kd, st, host_count=True)
    m.gather_queries(qd, st)
    cd = to_dev(c)
    if tiled:
        cd = m.tile_corpus(cd, st)
    sd = to_dev(sc) if sc is not None else None
    return w, m, c, sc, cd, sd, nu, st


def _snapshot(m, nu):
    torch.cuda.synchronize()
    return (m.topk_score[:nu].cpu().numpy().view(np.uint32).copy(),
            m.topk_index[:nu].cpu().numpy().copy())


@pytest.mark.parametrize("enc,tiled", [("bf16", False), ("fp8", False), ("bf16", True),
                                       ("fp8", True)])
def test_sequential_chunks_equal_one_batch(enc, tiled):
    # (sub-batches start at any query row, so the query tiling of each call
    # starts there too; tiled: the corpus in the tiled layout)
    w, m, c, sc, cd, sd, nu, st = _setup(enc=enc, tiled=tiled)
    m.score_chunked(cd, nu, nu, sd, st)
    s1, i1 = _snapshot(m, nu)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, w.q_req, c, w.k, scale=sc)
    for B in (1, 7, 32, 100, 128, 200):
        note(f"{enc}: chunks of {B}")
        m.topk_score.zero_()
        m.topk_index.zero_()
        m.score_chunked(cd, nu, B, sd, st)
        s2, i2 = _snapshot(m, nu)
        np.testing.assert_array_equal(i2, i1)
        np.testing.assert_array_equal(s2, s1)


@pytest.mark.parametrize("parts", [2, 3, 4])
def test_split_on_streams_equals_one_batch(parts):
    w, m, c, sc, cd, sd, nu, st = _setup()
    m.score_chunked(cd, nu, nu, sd, st)
    s1, i1 = _snapshot(m, nu)
    m.topk_score.zero_()
    m.topk_index.zero_()
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(parts)]   # default priority
    m.score_split(cd, nu, parts, streams, sd)
    s2, i2 = _snapshot(m, nu)
    np.testing.assert_array_equal(i2, i1)
    np.testing.assert_array_equal(s2, s1)


def test_max_unique_below_distinct_count_scores_every_group():
    """A batch limit B_r (max_unique) below the window's distinct count: the
    composition reads the count and scores the distinct queries in batches
    of at most B_r, so every request gets its result -- identical to the
    unlimited plan (and accepted by the oracle for a sample)."""
    import paper_2607_22578_amd as hs
    dev = device()
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    N = 9_000
    c, _ = synth.gaussian_rows(w.seed, synth.S_CORPUS, N, w.dim, "bf16")
    st = torch.cuda.current_stream(dev)
    kd, qd, cd = to_dev(w.keys), to_dev(w.q_req), to_dev(c)
    outs = []
    for cap in (0, 64, 200):
        m = hs.MergedRetrieval(w.R, w.dim, N, w.k, hs.HS_BF16, hs.HS_BF16, device=dev,
                               max_unique=cap)
        m.out_score.fill_(float("nan"))
        m.out_index.fill_(-7)
        m.run(kd, qd, cd, stream=st)
        torch.cuda.synchronize(dev)
        outs.append((m.out_score.cpu().numpy().view(np.uint32).copy(),
                     m.out_index.cpu().numpy().copy()))
        if cap:
            nu = int(m.n_unique.item())
            assert nu > cap   # the limit is really below the distinct count
            ref = check_dedup(m, w.keys)
            check_unique_topk(m, ref, w.q_req, c, w.k, sel=np.array([0, cap - 1, cap, nu - 1]))
    assert np.all(outs[0][1] >= 0)
    for s, i in outs[1:]:
        np.testing.assert_array_equal(i, outs[0][1])
        np.testing.assert_array_equal(s, outs[0][0])
