"""Parity of the rows beyond the window at the sizes the benchmark modes
time: cross-window reuse over the 1M-row corpus (a 4,096-entry store, three
successive windows; hit/miss split bit-exact against the store model, reused
rows bit-exact, a seeded sample of distinct queries per window under the
acceptance rule against the oracle), node signatures of 262,144 request
nodes (bit-exact), and micro-batching of the 1M-row window (sub-batches and
stream splits bit-identical to one batch)."""
import numpy as np
import pytest
import torch

from oracle import signature as sg
from oracle import store
import synth
from gpu_harness import check_dedup, check_delivery, check_unique_topk, device, note, to_dev

pytestmark = pytest.mark.gpu


def test_reuse_full_corpus():
    import paper_2607_22578_amd as hs
    dev = device()
    note("reuse: generating the 1M-row corpus")
    w0 = synth.make("ridge1m")
    wins = synth.window_stream("ridge1m", 3)
    m = hs.MergedRetrieval(w0.R, w0.dim, w0.n_corpus, w0.k, hs.HS_BF16, hs.HS_BF16, device=dev)
    m.enable_cache(4096)
    cd = to_dev(w0.corpus)
    st = torch.cuda.current_stream(dev)
    model = store.StoreModel(4096)
    last = {}
    rng = np.random.default_rng(17)
    for wi, win in enumerate(wins):
        m.run_cached(to_dev(win.keys), to_dev(win.q_req), cd, None, stream=st)
        torch.cuda.synchronize(dev)
        ref = check_dedup(m, win.keys)
        nu, uk = ref["n_unique"], ref["unique_keys"]
        mp_ref, nm = model.lookup(uk)
        np.testing.assert_array_equal(m.miss_pos[:nu].cpu().numpy().astype(np.int64), mp_ref)
        assert int(m.n_miss.item()) == nm
        ts = m.topk_score[:nu].cpu().numpy()
        ti = m.topk_index[:nu].cpu().numpy()
        hits = np.nonzero(mp_ref < 0)[0]
        for u in hits:
            s0, i0 = last[int(uk[u])]
            np.testing.assert_array_equal(ts[u].view(np.uint32), s0.view(np.uint32))
            np.testing.assert_array_equal(ti[u], i0)
        misses = np.nonzero(mp_ref >= 0)[0]
        for u in misses:
            last[int(uk[u])] = (ts[u].copy(), ti[u].copy())
        note(f"reuse window {wi}: {nu} distinct, {nm} misses, {len(hits)} hits bit-exact")
        sel = np.unique(np.concatenate([rng.choice(misses, size=min(4, len(misses)),
                                                   replace=False),
                                        rng.choice(hits, size=min(4, len(hits)), replace=False)
                                        if len(hits) else np.zeros(0, np.int64)]))
        check_unique_topk(m, ref, win.q_req, w0.corpus, w0.k, sel=sel)
        check_delivery(m, win.R)
        model.insert(uk, mp_ref, list(ts), list(ti))


def test_signatures_262k_nodes():
    import paper_2607_22578_amd as hs
    dev = device()
    cfg = synth.CONFIGS["ridge1m"]
    seed = synth.BASE_SEED + synth.ORDER.index("ridge1m")
    n = 262_144
    ranks = synth.zipf_ranks(seed, synth.S_ZIPF, cfg.n_templates, cfg.zipf_s, n)
    tids = synth.permutation(seed, synth.S_PERM, cfg.n_templates)[ranks]
    buf, off = synth.render_texts(seed, tids)
    note(f"signatures: {n} nodes, {buf.size} text bytes")
    op = np.full(n, 2, np.uint32)
    par = np.full(n, cfg.k, np.uint32).tobytes()
    poff = np.arange(n + 1, dtype=np.int64) * 4
    td = torch.from_numpy(buf).to(dev)
    dig = torch.empty((n, 32), dtype=torch.uint8, device=dev)
    keys = torch.empty(n, dtype=torch.int64, device=dev)
    hs.hs_signature(torch.from_numpy(op.view(np.int32)).to(dev), n, 0, n, dig, keys,
                    params=torch.from_numpy(np.frombuffer(par, np.uint8).copy()).to(dev),
                    param_off=torch.from_numpy(poff).to(dev), text=td,
                    text_off=torch.from_numpy(off).to(dev), flags=hs.HS_SIG_NORMALIZE_TEXT,
                    stream=torch.cuda.current_stream(dev))
    torch.cuda.synchronize(dev)
    rd, rk = sg.signatures(op, par, poff, buf.tobytes(), off, None, None, [(0, n)], True)
    np.testing.assert_array_equal(dig.cpu().numpy(), rd)
    np.testing.assert_array_equal(keys.cpu().numpy(), rk)
    assert len(np.unique(rk)) == len(np.unique(tids))


def test_batching_full_corpus():
    import paper_2607_22578_amd as hs
    dev = device()
    w = synth.make("ridge1m")
    m = hs.MergedRetrieval(w.R, w.dim, w.n_corpus, w.k, hs.HS_BF16, hs.HS_BF16, device=dev)
    st = torch.cuda.current_stream(dev)
    cd = to_dev(w.corpus)
    nu = m.dedup(to_dev(w.keys), st, host_count=True)
    m.gather_queries(to_dev(w.q_req), st)
    m.score_chunked(cd, nu, nu, None, st)
    torch.cuda.synchronize(dev)
    s1 = m.topk_score[:nu].cpu().numpy().view(np.uint32).copy()
    i1 = m.topk_index[:nu].cpu().numpy().copy()
    for B in (32, 128, 256):
        m.topk_index.zero_()
        m.score_chunked(cd, nu, B, None, st)
        torch.cuda.synchronize(dev)
        np.testing.assert_array_equal(m.topk_index[:nu].cpu().numpy(), i1)
        np.testing.assert_array_equal(m.topk_score[:nu].cpu().numpy().view(np.uint32), s1)
        note(f"batching: chunks of {B} identical")
    streams = [torch.cuda.Stream() for _ in range(2)]   # default priority
    m.topk_index.zero_()
    torch.cuda.synchronize(dev)
    m.score_split(cd, nu, 2, streams)
    torch.cuda.synchronize(dev)
    np.testing.assert_array_equal(m.topk_index[:nu].cpu().numpy(), i1)
    np.testing.assert_array_equal(m.topk_score[:nu].cpu().numpy().view(np.uint32), s1)
