"""Matrix-core scoring path on shapes away from the workload sizes, against
the oracle (acceptance rule of oracle/accept.py): dimensions that leave a
partial last K stage (the copies read zeros past d), corpora smaller than
one 384-row tile or with a ragged last tile, k-lists held in global memory
instead of LDS, k too large for the first-pass threshold seed, a seed that
samples several tiles per slice (k > 48) or one slice in two (a single
query tile over 256 slices), items of later rounds that start
from the order statistics of finished slices, and a merge with more
survivors than it ranks by counting (it sorts them)."""
import numpy as np
import pytest

import synth
from gpu_harness import check_dedup, check_delivery, check_unique_topk, note, run_merge

pytestmark = pytest.mark.gpu


def _stream(n_corpus: int, d: int, enc: str):
    """The 1M-row workload's request stream (329 distinct queries over 2,048
    requests) with query rows of width d and a fresh corpus of n_corpus rows
    in storage encoding `enc`."""
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    q, _ = synth.gaussian_rows(w.seed, synth.S_QUERY, 0, d, "bf16", row_ids=w.template_ids)
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, d, enc)
    return w, q, c, sc


@pytest.mark.parametrize("d,n_corpus", [(8, 1000), (40, 385), (200, 2000), (776, 1500)])
def test_bf16_partial_stage_and_ragged_tiles(d, n_corpus):
    w, q, c, _ = _stream(n_corpus, d, "bf16")
    note(f"bf16 d={d} N={n_corpus}")
    m = run_merge(w.keys, q, c, 10)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, q, c, 10)
    check_delivery(m, w.R)


@pytest.mark.parametrize("d,n_corpus", [(16, 700), (784, 2500)])
def test_fp8_partial_stage(d, n_corpus):
    w, q, c, sc = _stream(n_corpus, d, "fp8")
    note(f"fp8 d={d} N={n_corpus}")
    m = run_merge(w.keys, q, c, 10, scale=sc)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, q, c, 10, scale=sc)
    check_delivery(m, w.R)


@pytest.mark.parametrize("k", [18, 19, 64])
def test_lists_in_lds_and_global(k):
    # with a bf16 corpus, k-lists fit in LDS up to k = 18 and live in the
    # partial buffer in global memory from k = 19 on
    w, q, c, _ = _stream(6000, 768, "bf16")
    note(f"bf16 k={k}")
    m = run_merge(w.keys, q, c, k)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, q, c, k)
    check_delivery(m, w.R)


def test_k_beyond_seed():
    # 1,100 rows are three tiles, so the first pass sees at most 8 * 3 lane
    # maxima per query: fewer than k, and no threshold seed is written
    w, q, c, _ = _stream(1100, 128, "bf16")
    k = 300
    m = run_merge(w.keys, q, c, k)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, q, c, k)
    check_delivery(m, w.R)


def test_large_k_many_survivors():
    # k = 300 over 200,000 rows: fewer slices than k (no head cut), fewer lane
    # maxima than k (no seed) and no warm-up, so the cross-slice merge keeps
    # most of the 27 x 300 list keys and sorts them instead of ranking
    w, q, c, _ = _stream(200_000, 64, "bf16")
    k = 300
    note(f"bf16 k={k} N=200000 d=64")
    m = run_merge(w.keys, q, c, k)
    ref = check_dedup(m, w.keys)
    sel = np.random.default_rng(7).choice(ref["n_unique"], size=48, replace=False)
    check_unique_topk(m, ref, q, c, k, sel=np.sort(sel))
    check_delivery(m, w.R)


@pytest.mark.parametrize("enc", ["bf16", "fp8"])
def test_large_k_seed_samples_several_tiles(enc):
    # k = 100 over the 20M-row workload's request stream (2,197 distinct
    # queries: 18 query tiles, 14 slices on a 256-workgroup grid) and
    # 1,200,000 rows (3,125 tiles, 223 per slice): for k > 48 the seed pass
    # samples the first 223 / 16 = 13 tiles of every slice instead of one, so
    # the seed and the shared thresholds come from 13 x 14 x 8 lane maxima
    # per query
    w = synth.make("fp8_20m", n_corpus=1, with_corpus=False)
    d, n_corpus, k = 128, 1_200_000, 100
    q, _ = synth.gaussian_rows(w.seed, synth.S_QUERY, 0, d, "bf16", row_ids=w.template_ids)
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, d, enc)
    note(f"{enc} k={k} N={n_corpus} d={d}")
    m = run_merge(w.keys, q, c, k, scale=sc if enc == "fp8" else None)
    ref = check_dedup(m, w.keys)
    sel = np.random.default_rng(11).choice(ref["n_unique"], size=40, replace=False)
    check_unique_topk(m, ref, q, c, k, scale=sc if enc == "fp8" else None, sel=np.sort(sel))
    check_delivery(m, w.R)


@pytest.mark.parametrize("enc,k", [("bf16", 10), ("fp8", 10), ("bf16", 64)])
def test_seed_sample_every_second_slice(enc, k):
    # one query tile (the first 300 requests of the 1M-row stream, fewer than
    # 128 distinct) over 150,000 rows: 256 slices of one or two tiles, of
    # which the seed pass samples every second one (the others contribute
    # no lane maxima); bf16 with k = 64 keeps its lists in global memory
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    d, n_corpus = 64, 150_000
    keys = w.keys[:300]
    q, _ = synth.gaussian_rows(w.seed, synth.S_QUERY, 0, d, "bf16", row_ids=w.template_ids[:300])
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, d, enc)
    scale = sc if enc == "fp8" else None
    note(f"{enc} k={k} N={n_corpus} d={d}: seed sample of 128 of 256 slices")
    m = run_merge(keys, q, c, k, scale=scale)
    ref = check_dedup(m, keys)
    assert ref["n_unique"] <= 128
    check_unique_topk(m, ref, q, c, k, scale=scale)
    check_delivery(m, 300)


@pytest.mark.parametrize("enc", ["bf16", "fp8"])
def test_thresholds_from_finished_slices(enc):
    # k = 64 over 350,000 rows (912 tiles) for the 20M-row workload's request
    # stream (2,197 distinct queries, 18 query tiles): 71 slices of ~13 tiles,
    # 1,278 items in five rounds of the 256-workgroup grid, so items of
    # rounds 2-5 start from the order statistics that the finished slices
    # published (k-lists in global memory)
    w = synth.make("fp8_20m", n_corpus=1, with_corpus=False)
    d, n_corpus, k = 64, 350_000, 64
    q, _ = synth.gaussian_rows(w.seed, synth.S_QUERY, 0, d, "bf16", row_ids=w.template_ids)
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, d, enc)
    scale = sc if enc == "fp8" else None
    note(f"{enc} k={k} N={n_corpus} d={d}: five rounds")
    m = run_merge(w.keys, q, c, k, scale=scale)
    ref = check_dedup(m, w.keys)
    nu = ref["n_unique"]
    # eight queries of every query tile, and the first and last
    rng = np.random.default_rng(5)
    sel = [0, nu - 1]
    for b0 in range(0, nu, 128):
        sel.extend((b0 + rng.choice(min(128, nu - b0), size=8, replace=False)).tolist())
    check_unique_topk(m, ref, q, c, k, scale=scale, sel=np.unique(np.array(sel)))
    check_delivery(m, w.R)
