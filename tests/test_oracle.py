"""Pins for the oracle: each check ties it to something other than itself --
hand-derived worked examples, textbook library routines (numpy unique, fp64
matmul, lexsort, argmax, torch's fp8/bf16 dtypes), closed forms and brute
force on tiny inputs.  CPU only."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import accept

GOLD = os.path.join(os.path.dirname(__file__), "golden")
I64_MIN = np.iinfo(np.int64).min
I64_MAX = np.iinfo(np.int64).max


def _np_unique_ref(keys):
    u, first, inv, cnt = np.unique(keys, return_index=True, return_inverse=True,
                                   return_counts=True)
    return u, first.astype(np.int32), inv.astype(np.int32).ravel(), cnt.astype(np.int32)


# ---------------------------------------------------------------- dedup

def test_dedup_worked_example():
    g = json.load(open(os.path.join(GOLD, "dedup_worked.json")))
    keys = np.array([int(x) for x in g["keys"]], dtype=np.int64)
    r = oracle.dedup(keys)
    assert r["n_unique"] == len(g["unique_keys"])
    assert r["unique_keys"].tolist() == [int(x) for x in g["unique_keys"]]
    assert r["first_index"].tolist() == g["first_index"]
    assert r["counts"].tolist() == g["counts"]
    assert r["inverse"].tolist() == g["inverse"]


@pytest.mark.parametrize("seed", range(6))
def test_dedup_matches_numpy_unique(seed):
    rng = np.random.default_rng(seed)
    R = int(rng.integers(1, 3000))
    pool = int(rng.integers(1, 400))
    vals = rng.integers(I64_MIN, I64_MAX, size=pool, dtype=np.int64, endpoint=True)
    keys = vals[rng.integers(0, pool, size=R)]
    r = oracle.dedup(keys)
    u, first, inv, cnt = _np_unique_ref(keys)
    assert r["n_unique"] == len(set(keys.tolist())) == u.shape[0]
    np.testing.assert_array_equal(r["unique_keys"], u)
    np.testing.assert_array_equal(r["first_index"], first)
    np.testing.assert_array_equal(r["inverse"], inv)
    np.testing.assert_array_equal(r["counts"], cnt)
    assert int(r["counts"].sum()) == R
    # invariants: strictly increasing, U[inverse[i]] = key_i, first occurrence
    assert np.all(np.diff(r["unique_keys"]) > 0)
    np.testing.assert_array_equal(r["unique_keys"][r["inverse"]], keys)
    for u_, f in enumerate(r["first_index"]):
        assert keys[f] == r["unique_keys"][u_]
        assert not np.any(keys[:f] == keys[f])


@pytest.mark.parametrize("case", ["empty", "one", "all_equal", "all_distinct", "extremes",
                                  "negative"])
def test_dedup_edge_cases(case):
    if case == "empty":
        keys = np.zeros(0, np.int64)
    elif case == "one":
        keys = np.array([-17], np.int64)
    elif case == "all_equal":
        keys = np.full(777, 123456789, np.int64)
    elif case == "all_distinct":
        keys = np.random.default_rng(1).permutation(1000).astype(np.int64) * 3 - 1500
    elif case == "extremes":
        keys = np.array([I64_MAX, I64_MIN, 0, -1, I64_MAX, I64_MIN, 1], np.int64)
    else:
        keys = -np.arange(1, 50, dtype=np.int64)[::-1].repeat(2)
    r = oracle.dedup(keys)
    if keys.size == 0:
        assert r["n_unique"] == 0
        return
    u, first, inv, cnt = _np_unique_ref(keys)
    np.testing.assert_array_equal(r["unique_keys"], u)
    np.testing.assert_array_equal(r["first_index"], first)
    np.testing.assert_array_equal(r["inverse"], inv)
    np.testing.assert_array_equal(r["counts"], cnt)


# ---------------------------------------------------------------- decoding

def test_e4m3_decode_all_codes_vs_torch():
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.e4m3_decode(c) for c in range(256)])
    nan = np.isnan(ref)
    assert nan.sum() == 2 and np.isnan(got[nan]).all()      # 0x7F, 0xFF
    np.testing.assert_array_equal(got[~nan], ref[~nan])


def test_e4m3_decode_closed_forms():
    # values fixed by the OCP 8-bit float format definition (E4M3, bias 7)
    assert oracle.e4m3_decode(0x7E) == 448.0          # largest finite
    assert oracle.e4m3_decode(0x08) == 2.0 ** -6      # smallest normal
    assert oracle.e4m3_decode(0x01) == 2.0 ** -9      # smallest subnormal
    assert oracle.e4m3_decode(0x07) == 7 * 2.0 ** -9  # largest subnormal
    assert oracle.e4m3_decode(0x38) == 1.0            # e=7, m=0
    assert oracle.e4m3_decode(0x39) == 1.125
    assert oracle.e4m3_decode(0xB8) == -1.0
    assert oracle.e4m3_decode(0x80) == 0.0 and np.signbit(oracle.e4m3_decode(0x80))


def test_bf16_decode_vs_torch():
    bits = np.arange(0, 65536, 7, dtype=np.uint16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.bf16_decode(int(b)) for b in bits])
    fin = np.isfinite(ref)
    np.testing.assert_array_equal(got[fin], ref[fin])
    assert np.array_equal(np.isnan(got), np.isnan(ref))


# ---------------------------------------------------------------- scoring / top-k

def _decode_np(a, scale=None):
    """Independent numpy widening of storage encodings to float64."""
    if a.dtype == np.float32:
        return a.astype(np.float64)
    if a.dtype == np.uint16:
        return synth.bf16_bits_to_f32(a).astype(np.float64)
    t = torch.from_numpy(a.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    return t * scale.astype(np.float64)[:, None]


def _brute(Q, C, kk, scale=None):
    S = _decode_np(Q) @ _decode_np(C, scale).T     # fp64 library matmul
    n, N = S.shape
    sc = np.full((n, kk), -np.inf)
    ix = np.full((n, kk), -1, np.int64)
    for q in range(n):
        order = np.lexsort((np.arange(N), -S[q]))[:kk]
        sc[q, :len(order)] = S[q, order]
        ix[q, :len(order)] = order
    return S, sc, ix


def test_topk_worked_example():
    g = json.load(open(os.path.join(GOLD, "topk_worked.json")))
    C = np.array(g["corpus"], dtype=np.float32)
    for case in g["cases"]:
        Q = np.array([case["query"]], dtype=np.float32)
        s, i = oracle.topk_exact(Q, C, case["k"])
        want = np.array([float(x) for x in case["score"]])
        np.testing.assert_array_equal(s[0], want)
        assert i[0].tolist() == case["index"]


@pytest.mark.parametrize("enc", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("seed", [0, 1])
def test_topk_matches_bruteforce(enc, seed):
    rng = np.random.default_rng(seed)
    n, N, d, kk = 5, 300, 24, 12
    q_enc = "f32" if enc == "f32" else "bf16"
    Q, _ = synth.gaussian_rows(seed, 91, n, d, q_enc)
    C, sc = synth.gaussian_rows(seed, 92, N, d, enc)
    # plant exact duplicates of some rows at various positions
    for a, b in [(3, 250), (17, 18), (40, 299)]:
        C[b] = C[a]
        if sc is not None:
            sc[b] = sc[a]
    S, rs, ri = _brute(Q, C, kk, sc)
    for threads in (1, 3, 64):
        s, i = oracle.topk_exact(Q, C, kk, scale=sc, threads=threads)
        np.testing.assert_array_equal(i, ri)
        np.testing.assert_allclose(s, rs, rtol=1e-12, atol=1e-15)
    # exact scores of explicit pairs agree with the library matmul
    qi = rng.integers(0, n, 50)
    ci = rng.integers(0, N, 50)
    np.testing.assert_allclose(oracle.score_pairs(Q, C, qi, ci, scale=sc), S[qi, ci],
                               rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("threads", [1, 2, 64])
def test_topk_ties_straddling_rank_k(threads):
    # Groups of identical corpus rows whose scores tie exactly; one group is
    # planted so that it straddles rank k (its lower rows must be kept, in
    # ascending order), against the lexsort brute force.  Few queries and a
    # small corpus, with any thread count.
    d, N, kk = 16, 97, 7
    C, _ = synth.gaussian_rows(12, 90, N, d, "bf16")
    Q, _ = synth.gaussian_rows(12, 89, 3, d, "bf16")
    S0 = _decode_np(Q) @ _decode_np(C).T
    # the row ranked 5th for query 0 gets four copies spread over the corpus,
    # so ranks 5..8 tie and rank k = 7 cuts the group
    r5 = int(np.lexsort((np.arange(N), -S0[0]))[4])
    for b in (3, 50, 90):
        if b != r5:
            C[b] = C[r5]
    S, rs, ri = _brute(Q, C, kk)
    s, i = oracle.topk_exact(Q, C, kk, threads=threads)
    np.testing.assert_array_equal(i, ri)
    np.testing.assert_array_equal(s, rs)
    tied = sorted({r5, 3, 50, 90})
    assert i[0, 4:7].tolist() == tied[:3]
    assert s[0, 4] == s[0, 5] == s[0, 6]
    # one query and a corpus smaller than the thread count
    s1, i1 = oracle.topk_exact(Q[:1], C[:5], 9, threads=threads)
    _, rs1, ri1 = _brute(Q[:1], C[:5], 9)
    np.testing.assert_array_equal(i1, ri1)
    assert np.all(i1[0, 5:] == -1) and np.all(np.isneginf(s1[0, 5:]))


def test_unit_query_picks_column():
    # closed form: Q = e_j gives score(c) = C[c, j]
    d, N = 16, 200
    C, _ = synth.gaussian_rows(5, 93, N, d, "f32")
    for j in [0, 7, 15]:
        Q = np.zeros((1, d), np.float32)
        Q[0, j] = 1.0
        s, i = oracle.topk_exact(Q, C, N)
        col = C[:, j].astype(np.float64)
        np.testing.assert_array_equal(np.sort(s[0])[::-1], np.sort(col)[::-1])
        np.testing.assert_array_equal(s[0], col[i[0]])


def test_self_match_is_top1():
    # a corpus row equal to the (unit) query scores ||q||^2 and wins
    d, N = 32, 500
    C, _ = synth.gaussian_rows(6, 94, N, d, "f32")
    q = C[321:322].copy()
    s, i = oracle.topk_exact(q, C, 1)
    assert i[0, 0] == 321
    assert s[0, 0] == pytest.approx(float(np.sum(q.astype(np.float64) ** 2)), rel=1e-12)


def test_k1_is_first_argmax_and_k_equals_n_is_permutation():
    d, N = 8, 64
    C, _ = synth.gaussian_rows(7, 95, N, d, "bf16")
    C[50] = C[10]                    # a duplicate of some row
    Q, _ = synth.gaussian_rows(7, 96, 3, d, "bf16")
    S = _decode_np(Q) @ _decode_np(C).T
    s1, i1 = oracle.topk_exact(Q, C, 1)
    np.testing.assert_array_equal(i1[:, 0], np.argmax(S, axis=1))
    sN, iN = oracle.topk_exact(Q, C, N)
    for q in range(3):
        assert sorted(iN[q].tolist()) == list(range(N))
    sP, iP = oracle.topk_exact(Q, C, N + 5)
    assert np.all(iP[:, N:] == -1) and np.all(np.isneginf(sP[:, N:]))


def test_planted_tie_goes_to_lower_index():
    d, N = 16, 100
    C, _ = synth.gaussian_rows(8, 97, N, d, "bf16")
    Q = C[30:31].copy()
    C[77] = C[30]
    s, i = oracle.topk_exact(Q, C, 1)
    assert i[0, 0] == 30
    s, i = oracle.topk_exact(Q, C, 2)
    assert i[0].tolist() == [30, 77] and s[0, 0] == s[0, 1]


# ---------------------------------------------------------------- merged path

def test_merge_worked_example():
    g = json.load(open(os.path.join(GOLD, "topk_worked.json")))
    C = np.array(g["corpus"], dtype=np.float32)
    m = g["merge"]
    keys = np.array([int(x) for x in m["keys"]], np.int64)
    Q = np.array(m["queries"], dtype=np.float32)
    r = oracle.merge_retrieval(keys, Q, C, m["k"])
    assert r["n_unique"] == m["n_unique"]
    np.testing.assert_array_equal(r["out_score"], np.array(m["out_score"], np.float32))
    np.testing.assert_array_equal(r["out_index"], np.array(m["out_index"]))


def test_merged_equals_independent_tiny():
    w = synth.make("tiny")
    r = oracle.merge_retrieval(w.keys, w.q_req, w.corpus, w.k)
    assert r["n_unique"] == len(set(w.keys.tolist())) == 20
    assert int(r["counts"].sum()) == w.R
    # independent retrieval for every request, no dedup
    s, i = oracle.topk_exact(w.q_req, w.corpus, w.k)
    np.testing.assert_array_equal(r["out_index"], i.astype(np.int32))
    np.testing.assert_array_equal(r["out_score"], s.astype(np.float32))
    # and against a brute force of the whole thing
    S, bs, bi = _brute(w.q_req, w.corpus, w.k)
    np.testing.assert_array_equal(r["out_index"], bi)


def test_merged_subset_selection():
    w = synth.make("ridge1m", n_corpus=2000)
    full = oracle.merge_retrieval(w.keys, w.q_req, w.corpus, w.k)
    sel = np.array([0, 5, full["n_unique"] - 1], np.int64)
    part = oracle.merge_retrieval(w.keys, w.q_req, w.corpus, w.k, u_sel=sel)
    np.testing.assert_array_equal(part["u_index"], full["u_index"][sel])
    hit = np.isin(full["inverse"], sel)
    np.testing.assert_array_equal(part["out_index"][hit], full["out_index"][hit])
    assert np.all(part["out_index"][~hit] == -2)


def test_gather_rows_matches_fancy_indexing():
    rng = np.random.default_rng(3)
    src = rng.integers(0, 65535, size=(100, 40), dtype=np.uint16)
    for idx in [rng.integers(0, 100, 57).astype(np.int32), rng.integers(0, 100, 9)]:
        np.testing.assert_array_equal(oracle.gather_rows(src, idx), src[idx])
    with pytest.raises(IndexError):
        oracle.gather_rows(src, np.array([100], np.int32))


# ---------------------------------------------------------------- acceptance rule

def _accept_case():
    d, N, k = 16, 400, 10
    Q, _ = synth.gaussian_rows(11, 98, 4, d, "f32")
    C, _ = synth.gaussian_rows(11, 99, N, d, "f32")
    rs, ri = oracle.topk_exact(Q, C, k + 1)
    return Q, C, N, k, rs, ri


def test_accept_rule_passes_exact_and_rejects_mistakes():
    Q, C, N, k, rs, ri = _accept_case()
    gs = rs[:, :k].astype(np.float32)
    gi = ri[:, :k].copy()
    ex = rs[:, :k]
    assert accept.check_all(gs, gi, rs, ri, ex, N, k) == []
    # a wrong index (rank k+1 instead of rank 1) is caught
    bad_i = gi.copy()
    bad_i[0, 0] = ri[0, k]
    ex_bad = ex.copy()
    ex_bad[0, 0] = rs[0, k]
    assert accept.check_all(gs, bad_i, rs, ri, ex_bad, N, k)
    # a score off by 1% is caught
    bad_s = gs.copy()
    bad_s[1, 3] *= 1.01
    assert accept.check_all(bad_s, gi, rs, ri, ex, N, k)
    # swapped order is caught
    sw_s, sw_i = gs.copy(), gi.copy()
    sw_s[2, [0, 1]] = sw_s[2, [1, 0]]
    sw_i[2, [0, 1]] = sw_i[2, [1, 0]]
    assert accept.check_all(sw_s, sw_i, rs, ri, ex[:, :][:, :], N, k)
    # a result computed against the negated query (sign mistake) is caught
    ns, ni = oracle.topk_exact(-Q, C, k)
    ex_n = oracle.score_pairs(Q, C, np.repeat(np.arange(4), k), ni.ravel()).reshape(4, k)
    assert accept.check_all(-ns.astype(np.float32), ni, rs, ri, ex_n, N, k)
