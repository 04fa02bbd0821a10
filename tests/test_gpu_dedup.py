"""Dedup on the GPU, bit-exact against the oracle."""
import zlib

import numpy as np
import pytest
import torch

import synth
from gpu_harness import device, note

pytestmark = pytest.mark.gpu

I64_MIN = np.iinfo(np.int64).min
I64_MAX = np.iinfo(np.int64).max


def _gpu_dedup(keys, host_count=False):
    import paper_2607_22578_amd as hs
    import oracle
    dev = device()
    R = keys.shape[0]
    plan = hs.hs_merge_plan(R, 8, 1, 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    R1 = max(R, 1)
    kd = torch.from_numpy(keys.astype(np.int64)).to(dev) if R else None
    uk = torch.full((R1,), 7, dtype=torch.int64, device=dev)
    fi = torch.full((R1,), -7, dtype=torch.int32, device=dev)
    ct = torch.full((R1,), -7, dtype=torch.int32, device=dev)
    inv = torch.full((R1,), -7, dtype=torch.int32, device=dev)
    nu = torch.full((1,), -7, dtype=torch.int64, device=dev)
    st = torch.cuda.current_stream(dev)
    nh = hs.hs_dedup(plan, kd, uk, fi, ct, inv, nu, True if host_count else None, ws, stream=st)
    torch.cuda.synchronize(dev)
    ref = oracle.dedup(keys)
    n = int(nu.item())
    assert n == ref["n_unique"]
    if host_count:
        assert nh == n
    np.testing.assert_array_equal(uk[:n].cpu().numpy(), ref["unique_keys"])
    np.testing.assert_array_equal(fi[:n].cpu().numpy(), ref["first_index"])
    np.testing.assert_array_equal(ct[:n].cpu().numpy(), ref["counts"])
    np.testing.assert_array_equal(inv[:R].cpu().numpy(), ref["inverse"])
    return uk[:n].cpu().numpy(), inv[:R].cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "ridge1m", "mfma4m", "fp8_20m", "dedup256k"])
def test_dedup_workload_keys(name):
    w = synth.make(name, with_corpus=False)
    note(f"dedup {name} R={w.R}")
    _gpu_dedup(w.keys, host_count=(name == "ridge1m"))


@pytest.mark.parametrize("case", ["one", "two_equal", "all_equal_small", "all_equal_radix",
                                  "distinct_small", "distinct_radix", "extremes_small",
                                  "extremes_radix", "negative", "boundary_4096",
                                  "boundary_4097", "ragged_radix", "narrow_range_radix",
                                  "wide_and_narrow", "all_min_hash", "distinct_hash",
                                  "boundary_2048", "boundary_2049", "high_bits_hash",
                                  "dense_span_r_minus_1", "radix_span_r", "dense_negative",
                                  "dense_hot_zipf"])
def test_dedup_edge_cases(case):
    # paths: hash table up to 2,048 keys, bitonic sort up to 4,096, radix sort
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    if case == "one":
        keys = np.array([12345], np.int64)
    elif case == "two_equal":
        keys = np.array([-3, -3], np.int64)
    elif case == "all_equal_small":
        keys = np.full(3000, I64_MIN, np.int64)
    elif case == "all_equal_radix":
        keys = np.full(50_000, 42, np.int64)
    elif case == "distinct_small":
        keys = rng.permutation(4000).astype(np.int64) * 7919 - 10 ** 6
    elif case == "distinct_radix":
        keys = rng.integers(I64_MIN, I64_MAX, size=70_000, dtype=np.int64, endpoint=True)
    elif case == "extremes_small":
        keys = rng.choice(np.array([I64_MIN, I64_MAX, 0, -1, 1], np.int64), size=1000)
    elif case == "extremes_radix":
        keys = rng.choice(np.array([I64_MIN, I64_MAX, 0, -1, 1, I64_MIN + 1], np.int64),
                          size=9000)
    elif case == "negative":
        keys = -rng.integers(1, 500, size=6000).astype(np.int64)
    elif case == "boundary_4096":
        keys = rng.integers(0, 1000, size=4096).astype(np.int64)
    elif case == "boundary_4097":
        keys = rng.integers(0, 1000, size=4097).astype(np.int64)
    elif case == "all_min_hash":              # only the key that maps to 0
        keys = np.full(2048, I64_MIN, np.int64)
    elif case == "distinct_hash":
        keys = rng.integers(I64_MIN, I64_MAX, size=2048, dtype=np.int64, endpoint=True)
    elif case == "boundary_2048":
        keys = rng.integers(-50, 50, size=2048).astype(np.int64)
    elif case == "boundary_2049":
        keys = rng.integers(-50, 50, size=2049).astype(np.int64)
    elif case == "high_bits_hash":            # keys that differ only in their top bits
        keys = (rng.integers(0, 4096, size=1500).astype(np.int64) << 52)
    elif case == "ragged_radix":
        keys = rng.integers(-2 ** 40, 2 ** 40, size=3 * 4096 + 77).astype(np.int64)
    elif case == "dense_span_r_minus_1":      # R values exactly: direct addressing
        keys = (rng.permutation(9000) + 777).astype(np.int64)
    elif case == "radix_span_r":              # one value more than R: the sort
        keys = (rng.permutation(9001)[:9000] + 777).astype(np.int64)
        keys[0], keys[1] = 777, 777 + 9000
    elif case == "dense_negative":            # a narrow span around zero
        keys = rng.integers(-3000, 3000, size=20_000).astype(np.int64)
    elif case == "dense_hot_zipf":            # one key in half the requests
        keys = rng.integers(0, 50_000, size=100_000).astype(np.int64)
        keys[rng.random(100_000) < 0.5] = 31_337
    elif case == "narrow_range_radix":        # 18-bit span, far from zero
        keys = (rng.integers(0, 200_000, size=100_000) + 2 ** 50).astype(np.int64)
    else:                                     # one outlier forces all 64 bits
        keys = rng.integers(0, 300, size=20_000).astype(np.int64)
        keys[12345] = I64_MIN
    _gpu_dedup(keys)


def test_dedup_empty():
    _gpu_dedup(np.zeros(0, np.int64))


def test_dedup_deterministic():
    w = synth.make("mfma4m", with_corpus=False)
    a = _gpu_dedup(w.keys)
    b = _gpu_dedup(w.keys)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


@pytest.mark.parametrize("case", ["dense", "radix"])
def test_dedup_more_tiles_than_workgroups(case):
    # over 8M keys: 2,052 tiles of 4,096 keys, more than the prep launch
    # (1,024) and the persistent sort (at most 256) have workgroups, so each
    # takes several tiles; 8,193 value blocks in the dense scan's look-back
    # chain; direct addressing (keys over a span below R) and the radix sort
    rng = np.random.default_rng(5 if case == "dense" else 6)
    R = (1 << 23) + 12_345
    if case == "dense":
        keys = rng.integers(-(1 << 22), 1 << 22, size=R).astype(np.int64)
    else:
        keys = rng.integers(0, 1 << 40, size=R).astype(np.int64)
        keys[rng.random(R) < 0.3] = 17   # a hot key
    note(f"dedup {case} R={R}")
    _gpu_dedup(keys)


@pytest.mark.parametrize("tiles", [64, 65, 257])
def test_radix_digit_offsets_around_the_tile_threshold(tiles):
    # the sort takes its digit offsets straight from the histogram up to 64
    # tiles of 4,096 keys and from per-digit row scans above; 257 tiles is
    # more than the persistent sort's 256 workgroups (one takes two tiles);
    # ragged last tile, hot keys, negative keys
    rng = np.random.default_rng(100 + tiles)
    R = tiles * 4096 - 1000
    keys = rng.integers(-(1 << 62), 1 << 62, size=R).astype(np.int64)
    keys[rng.random(R) < 0.2] = -5
    keys[rng.random(R) < 0.1] = 1 << 61
    note(f"dedup radix R={R} ({tiles} tiles)")
    _gpu_dedup(keys)


def test_dense_and_sort_paths_alternate_on_one_workspace():
    # the same plan and workspace for a dense-range batch, then a sort-path
    # batch, then dense again: every launch resets the scratch it needs
    rng = np.random.default_rng(77)
    R = 40_000
    dense = rng.integers(0, R // 2, size=R).astype(np.int64)
    wide = rng.integers(-(1 << 40), 1 << 40, size=R).astype(np.int64)
    for k in (dense, wide, dense, wide):
        _gpu_dedup(k)


def test_sort_path_beside_a_concurrent_score_call():
    # the sort runs as one persistent launch whose workgroups wait for each
    # other at grid barriers; a score call on a second stream (a persistent
    # grid of its own, one workgroup on every CU) runs at the same time: both
    # finish and both are exact
    import oracle
    import paper_2607_22578_amd as hs
    from gpu_harness import check_dedup, check_unique_topk, to_dev
    dev = device()
    w = synth.make("ridge1m", n_corpus=1, with_corpus=False)
    N = 400_000   # a score call of ~0.3 ms, longer than the sort
    c, _ = synth.gaussian_rows(w.seed, synth.S_CORPUS, N, w.dim, "bf16")
    m = hs.MergedRetrieval(w.R, w.dim, N, w.k, hs.HS_BF16, hs.HS_BF16, device=dev)
    st = torch.cuda.current_stream(dev)
    cd = to_dev(c)
    nu = m.dedup(to_dev(w.keys), st, host_count=True)
    m.gather_queries(to_dev(w.q_req), st)
    torch.cuda.synchronize(dev)
    ref_w = check_dedup(m, w.keys)

    rng = np.random.default_rng(31)
    R = 300_000
    keys = rng.integers(-(1 << 50), 1 << 50, size=R).astype(np.int64)
    keys[rng.random(R) < 0.25] = 12345
    ref = oracle.dedup(keys)
    plan = hs.hs_merge_plan(R, 8, 1, 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    kdev = torch.from_numpy(keys).to(dev)
    uk = torch.empty(R, dtype=torch.int64, device=dev)
    fi = torch.empty(R, dtype=torch.int32, device=dev)
    ct = torch.empty(R, dtype=torch.int32, device=dev)
    inv = torch.empty(R, dtype=torch.int32, device=dev)
    n_dev = torch.empty(1, dtype=torch.int64, device=dev)
    other = torch.cuda.Stream(dev)   # default priority
    for rep in range(3):
        note(f"concurrent sort + score, repetition {rep}")
        m.topk_score.zero_()
        m.topk_index.zero_()
        torch.cuda.synchronize(dev)
        m.score_chunked(cd, nu, nu, None, other)
        hs.hs_dedup(plan, kdev, uk, fi, ct, inv, n_dev, None, ws, stream=st)
        torch.cuda.synchronize(dev)
        n = int(n_dev.item())
        assert n == ref["n_unique"]
        np.testing.assert_array_equal(uk[:n].cpu().numpy(), ref["unique_keys"])
        np.testing.assert_array_equal(fi[:n].cpu().numpy(), ref["first_index"])
        np.testing.assert_array_equal(ct[:n].cpu().numpy(), ref["counts"])
        np.testing.assert_array_equal(inv.cpu().numpy(), ref["inverse"])
        check_unique_topk(m, ref_w, w.q_req, c, w.k, sel=np.array([0, nu // 2, nu - 1]))
