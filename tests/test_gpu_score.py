"""Score + top-k + delivery on the GPU against the oracle (acceptance rule of
oracle/accept.py), at sizes the oracle finishes in seconds that still span
several tiles, several query tiles and ragged tails."""
import numpy as np
import pytest
import torch

import synth
from gpu_harness import (check_dedup, check_delivery, check_requests_vs_oracle,
                         check_unique_topk, device, note, run_merge, to_dev)

pytestmark = pytest.mark.gpu


def _full_check(w, corpus, scale=None, mode="device", sample_requests=64):
    note(f"{w.cfg.name}: R={w.R} N={corpus.shape[0]} d={w.dim} k={w.k} mode={mode}")
    m = run_merge(w.keys, w.q_req, corpus, w.k, scale=scale, n_unique_mode=mode)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, w.q_req, corpus, w.k, scale=scale)
    check_delivery(m, w.R)
    rng = np.random.default_rng(0)
    reqs = rng.choice(w.R, size=min(sample_requests, w.R), replace=False)
    check_requests_vs_oracle(m, ref, reqs, w.q_req, corpus, w.k, scale=scale)
    return m, ref


def test_tiny_fp32_full_path():
    w = synth.make("tiny")
    _full_check(w, w.corpus, sample_requests=w.R)


@pytest.mark.parametrize("mode", ["device", "host"])
def test_ridge_shape_reduced_corpus(mode):
    # 329 distinct queries = 3 query tiles (last one partial); 20,000 rows =
    # 156 full tiles + a ragged one
    w = synth.make("ridge1m", n_corpus=20_000)
    _full_check(w, w.corpus, mode=mode)


def test_fp32_multi_query_tiles_ragged():
    cfg_w = synth.make("ridge1m", n_corpus=3_001, with_corpus=False)
    # fp32 variant of the same request stream: 329 distinct queries
    q, _ = synth.gaussian_rows(cfg_w.seed, synth.S_QUERY, 0, 384, "f32",
                               row_ids=cfg_w.template_ids)
    c, _ = synth.gaussian_rows(cfg_w.seed, synth.S_CORPUS, 3_001, 384, "f32")
    m = run_merge(cfg_w.keys, q, c, 10)
    ref = check_dedup(m, cfg_w.keys)
    check_unique_topk(m, ref, q, c, 10)
    check_delivery(m, cfg_w.R)


@pytest.mark.parametrize("k", [1, 32, 33, 100])
def test_fp32_k_values(k):
    # k <= 32: lists in LDS merged by one wave per query (sorted lists);
    # k > 32: lists in the workspace, one thread per query; 329 distinct
    # queries over 5,003 rows (6 query tiles, the last with 9 live queries)
    cfg_w = synth.make("ridge1m", n_corpus=5_003, with_corpus=False)
    q, _ = synth.gaussian_rows(cfg_w.seed, synth.S_QUERY, 0, 384, "f32",
                               row_ids=cfg_w.template_ids)
    c, _ = synth.gaussian_rows(cfg_w.seed, synth.S_CORPUS, 5_003, 384, "f32")
    note(f"fp32 k={k}")
    m = run_merge(cfg_w.keys, q, c, k)
    ref = check_dedup(m, cfg_w.keys)
    check_unique_topk(m, ref, q, c, k)
    check_delivery(m, cfg_w.R)


@pytest.mark.parametrize("d", [4, 36, 96, 100])
@pytest.mark.parametrize("k", [10, 40])
def test_fp32_odd_widths(d, k):
    # widths whose 32-wide K chunks are odd in number (d = 96: three) or end in
    # a partial chunk (d = 4, 36, 100), so the two-ahead K prefetch takes its
    # mid-loop exit and its zero-filled last chunk; k <= 32 (one wave per query
    # ranks a tile with its list) and k > 32 (lists in the workspace); a ragged
    # corpus of 2,999 rows (the last 64-row tile partial)
    cfg_w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    ids = cfg_w.template_ids[:300]
    keys = cfg_w.keys[:300]
    q, _ = synth.gaussian_rows(cfg_w.seed, synth.S_QUERY, 0, d, "f32", row_ids=ids)
    c, _ = synth.gaussian_rows(cfg_w.seed, synth.S_CORPUS, 2_999, d, "f32")
    note(f"fp32 d={d} k={k}")
    m = run_merge(keys, q, c, k)
    ref = check_dedup(m, keys)
    check_unique_topk(m, ref, q, c, k)
    check_delivery(m, len(keys))


@pytest.mark.parametrize("k", [1, 32, 100])
def test_k_values(k):
    w = synth.make("ridge1m", n_corpus=9_000)
    m = run_merge(w.keys, w.q_req, w.corpus, k)
    ref = check_dedup(m, w.keys)
    check_unique_topk(m, ref, w.q_req, w.corpus, k)
    check_delivery(m, w.R)


@pytest.mark.parametrize("tiled", [False, True])
@pytest.mark.parametrize("N", [0, 1, 7, 129])
def test_k_exceeds_corpus_pads(N, tiled):
    w = synth.make("ridge1m", n_corpus=max(N, 1))
    corpus = w.corpus[:N]
    k = 10
    m = run_merge(w.keys, w.q_req, corpus, k, tiled=tiled)
    ref = check_dedup(m, w.keys)
    if N > 0:
        check_unique_topk(m, ref, w.q_req, corpus, k)
    nu = ref["n_unique"]
    gi = m.topk_index[:nu].cpu().numpy()
    gs = m.topk_score[:nu].cpu().numpy()
    if N < k:
        assert np.all(gi[:, N:] == -1) and np.all(np.isneginf(gs[:, N:]))
    if N > 0:
        assert np.all(np.sort(gi[:, :min(N, k)], axis=1) >= 0)
    check_delivery(m, w.R)


def test_planted_ties_lower_index_wins():
    """Identical corpus rows give bit-identical scores; the lower row comes
    first, and is the one kept when the tie straddles rank k."""
    import oracle
    w = synth.make("ridge1m", n_corpus=40_000)
    C = w.corpus.copy()
    ref = oracle.dedup(w.keys)
    k = w.k
    rows = ref["first_index"][:6].astype(np.int64)
    rs, ri = oracle.topk_exact(w.q_req, C, k, q_rows=rows)
    planted = []
    # query 0: tie at rank 1 -> copy r_1 to a later row in another tile/slice
    a = int(ri[0, 0]); b = 39_990 if a < 39_990 else 5
    C[b] = C[a]; planted.append((0, min(a, b), max(a, b), "both"))
    # query 1: tie straddling rank k -> copy r_k to a higher row
    a = int(ri[1, k - 1]); b = 39_000 if a < 39_000 else 3
    C[b] = C[a]; planted.append((1, min(a, b), max(a, b), "lower_only"))
    m = run_merge(w.keys, w.q_req, C, k)
    check_dedup(m, w.keys)
    check_unique_topk(m, ref, w.q_req, C, k, sel=np.arange(6))
    gi = m.topk_index[:6].cpu().numpy()
    gs = m.topk_score[:6].cpu().numpy()
    for u, lo, hi, kind in planted:
        row = gi[u].tolist()
        if kind == "both":
            assert lo in row and hi in row and row.index(lo) + 1 == row.index(hi), row
            assert gs[u, row.index(lo)] == gs[u, row.index(hi)]
        else:
            # after planting, oracle's rank-k entry is the lower copy; the
            # higher copy ranks k+1 and must be excluded
            rs2, ri2 = oracle.topk_exact(w.q_req, C, k + 1, q_rows=rows[u:u + 1])
            if ri2[0, k - 1] == lo and ri2[0, k] == hi:
                assert lo in row and hi not in row, row


def test_fp8_corpus_all_codes():
    """fp8 e4m3 corpus with per-row scales; one row holds every finite code."""
    w = synth.make("fp8_20m", n_corpus=12_345)
    C = w.corpus.copy()
    S = w.scale.copy()
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    C[100] = np.resize(codes, C.shape[1])
    C[7_000] = np.resize(codes[::-1], C.shape[1])
    S[100] = 1.0 / 448.0
    _full_check(w, C, scale=S)


def test_deterministic_repeat():
    w = synth.make("ridge1m", n_corpus=15_000)
    m1 = run_merge(w.keys, w.q_req, w.corpus, w.k)
    m2 = run_merge(w.keys, w.q_req, w.corpus, w.k)
    nu = int(m1.n_unique.item())
    assert torch.equal(m1.topk_index[:nu], m2.topk_index[:nu])
    assert torch.equal(m1.topk_score[:nu].view(torch.int32), m2.topk_score[:nu].view(torch.int32))
    assert torch.equal(m1.out_index, m2.out_index)
