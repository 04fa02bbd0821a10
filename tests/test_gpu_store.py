"""Cross-window result reuse on the device (hs_cache_* with the whole path,
MergedRetrieval.run_cached) against the oracle's store model: per window,
the hit/miss split and miss numbering bit-exactly, reused rows bit-exactly
equal to the rows the device computed when the key was last missed, every
distinct query's row under the acceptance rule against a fresh oracle
retrieval, and delivery to every request."""
import numpy as np
import pytest
import torch

import oracle
from oracle import store
import synth
from gpu_harness import check_dedup, check_delivery, check_unique_topk, device, enc_code, note, \
    to_dev

pytestmark = pytest.mark.gpu

N_CORPUS = 12_000     # 31 full 384-row tiles and a ragged one


def _run(capacity, n_windows, k=10, enc="bf16", n_corpus=N_CORPUS, workload="ridge1m",
         n_check=None, tiled=False):
    import paper_2607_22578_amd as hs
    dev = device()
    wins = synth.window_stream(workload, n_windows)
    d = wins[0].dim
    c, sc = synth.gaussian_rows(wins[0].seed, synth.S_CORPUS, n_corpus, d, enc)
    R = wins[0].R
    m = hs.MergedRetrieval(R, d, n_corpus, k, enc_code(wins[0].q_req), enc_code(c), device=dev,
                           tiled_corpus=tiled)
    m.enable_cache(capacity)
    cd = to_dev(c)
    sd = to_dev(sc) if sc is not None else None
    st = torch.cuda.current_stream(dev)
    if tiled:
        cd = m.tile_corpus(cd, st)
    model = store.StoreModel(capacity)
    last = {}          # key -> (scores, indices) the device computed at its last miss
    n_hits = []
    for w, win in enumerate(wins):
        note(f"store C={capacity} enc={enc} k={k} window {w}")
        kd, qd = to_dev(win.keys), to_dev(win.q_req)
        m.run_cached(kd, qd, cd, sd, stream=st)
        torch.cuda.synchronize(dev)
        ref = check_dedup(m, win.keys)
        nu = ref["n_unique"]
        uk = ref["unique_keys"]
        mp_ref, nm_ref = model.lookup(uk)
        mp = m.miss_pos[:nu].cpu().numpy().astype(np.int64)
        np.testing.assert_array_equal(mp, mp_ref)
        assert int(m.n_miss.item()) == nm_ref
        np.testing.assert_array_equal(m.miss_first[:nm_ref].cpu().numpy(),
                                      ref["first_index"][mp_ref >= 0])
        ts = m.topk_score[:nu].cpu().numpy()
        ti = m.topk_index[:nu].cpu().numpy()
        for u in np.nonzero(mp_ref < 0)[0]:
            s0, i0 = last[int(uk[u])]
            np.testing.assert_array_equal(ts[u].view(np.uint32), s0.view(np.uint32))
            np.testing.assert_array_equal(ti[u], i0)
        for u in np.nonzero(mp_ref >= 0)[0]:
            last[int(uk[u])] = (ts[u].copy(), ti[u].copy())
        sel = None
        if n_check is not None:   # a seeded sample of hits and misses
            rng = np.random.default_rng(w)
            sel = np.sort(rng.choice(nu, size=min(n_check, nu), replace=False))
        check_unique_topk(m, ref, win.q_req, c, k, scale=sc, sel=sel)
        check_delivery(m, R)
        model.insert(uk, mp_ref, list(ts), list(ti))
        n_hits.append(int((mp_ref < 0).sum()))
    return n_hits


def test_reuse_across_windows():
    hits = _run(4096, 3)
    assert hits[0] == 0 and hits[1] > 0 and hits[2] > 0


def test_small_store_with_shared_entries():
    hits = _run(64, 3)
    assert hits[0] == 0 and hits[1] > 0


def test_one_entry_store():
    _run(1, 3)


def test_fp8_corpus_and_global_lists():
    _run(1024, 2, k=40, enc="fp8")


@pytest.mark.parametrize("enc", ["bf16", "fp8"])
def test_reuse_on_the_tiled_corpus(enc):
    # the store with the corpus in the tiled layout, as the benchmark runs it
    hits = _run(4096, 3, enc=enc, tiled=True)
    assert hits[0] == 0 and hits[1] > 0


def test_first_window_equals_uncached_path():
    # with an empty store every key misses and is scored in the same order,
    # so the cached path must reproduce the plain path bit for bit
    import paper_2607_22578_amd as hs
    dev = device()
    win = synth.window_stream("ridge1m", 1)[0]
    c, _ = synth.gaussian_rows(win.seed, synth.S_CORPUS, N_CORPUS, win.dim, "bf16")
    cd, kd, qd = to_dev(c), to_dev(win.keys), to_dev(win.q_req)
    st = torch.cuda.current_stream(dev)
    a = hs.MergedRetrieval(win.R, win.dim, N_CORPUS, 10, hs.HS_BF16, hs.HS_BF16, device=dev)
    b = hs.MergedRetrieval(win.R, win.dim, N_CORPUS, 10, hs.HS_BF16, hs.HS_BF16, device=dev)
    b.enable_cache(2048)
    a.run(kd, qd, cd, stream=st)
    b.run_cached(kd, qd, cd, stream=st)
    torch.cuda.synchronize(dev)
    np.testing.assert_array_equal(a.out_index.cpu().numpy(), b.out_index.cpu().numpy())
    np.testing.assert_array_equal(a.out_score.cpu().numpy().view(np.uint32),
                                  b.out_score.cpu().numpy().view(np.uint32))


def test_reset_empties_the_store():
    import paper_2607_22578_amd as hs
    dev = device()
    wins = synth.window_stream("ridge1m", 2)
    c, _ = synth.gaussian_rows(wins[0].seed, synth.S_CORPUS, 2000, wins[0].dim, "bf16")
    cd = to_dev(c)
    st = torch.cuda.current_stream(dev)
    m = hs.MergedRetrieval(wins[0].R, wins[0].dim, 2000, 10, hs.HS_BF16, hs.HS_BF16, device=dev)
    m.enable_cache(4096)
    m.run_cached(to_dev(wins[0].keys), to_dev(wins[0].q_req), cd, stream=st)
    hs.hs_cache_reset(m.plan, m.cache, m.cache_capacity, stream=st)
    m.run_cached(to_dev(wins[1].keys), to_dev(wins[1].q_req), cd, stream=st)
    torch.cuda.synchronize(dev)
    nu = int(m.n_unique.item())
    assert int(m.n_miss.item()) == nu
    assert (m.miss_pos[:nu].cpu().numpy() == np.arange(nu)).all()


def test_repeated_window_all_hits():
    # a store large enough that no two of the window's keys share an entry:
    # the second pass over the same window misses nothing (no scoring work)
    C = 1 << 20
    win = synth.window_stream("ridge1m", 1)[0]
    assert len({store.entry_of(int(x), C) for x in np.unique(win.keys)}) == \
        len(np.unique(win.keys))
    import paper_2607_22578_amd as hs
    dev = device()
    c, _ = synth.gaussian_rows(win.seed, synth.S_CORPUS, 3000, win.dim, "bf16")
    cd, kd, qd = to_dev(c), to_dev(win.keys), to_dev(win.q_req)
    st = torch.cuda.current_stream(dev)
    m = hs.MergedRetrieval(win.R, win.dim, 3000, 10, hs.HS_BF16, hs.HS_BF16, device=dev)
    m.enable_cache(C)
    m.run_cached(kd, qd, cd, stream=st)
    torch.cuda.synchronize(dev)
    s1, i1 = m.out_score.clone(), m.out_index.clone()
    m.run_cached(kd, qd, cd, stream=st)
    torch.cuda.synchronize(dev)
    assert int(m.n_miss.item()) == 0
    nu = int(m.n_unique.item())
    assert (m.miss_pos[:nu] == -1).all()
    assert torch.equal(m.out_index, i1)
    assert torch.equal(m.out_score.view(torch.int32), s1.view(torch.int32))


def test_many_distinct_keys():
    # 32,768 requests per window (~10k distinct): the store's multi-workgroup
    # insert path, k = 32
    hits = _run(16384, 2, k=32, n_corpus=3000, workload="mfma4m", n_check=64)
    assert hits[0] == 0 and hits[1] > 0

