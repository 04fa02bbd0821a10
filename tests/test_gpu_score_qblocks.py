"""Matrix-core scoring with query tiles whose queries fill 1, 2, 3 or 4 of
the tile's 32-query blocks (the kernel skips the empty blocks), against the
oracle (acceptance rule of oracle/accept.py): distinct-query counts on both
sides of every block boundary, bf16 and fp8 corpora, k-lists in LDS and in
global memory."""
import numpy as np
import pytest

import synth
from gpu_harness import check_dedup, check_delivery, check_unique_topk, note, run_merge

pytestmark = pytest.mark.gpu


def _requests(n_distinct: int, d: int, seed: int = 11):
    # 3 requests per distinct query, shuffled; query rows drawn per template
    rng = np.random.default_rng(seed + n_distinct)
    tids = rng.permutation(np.repeat(np.arange(n_distinct, dtype=np.int64), 3))
    keys = synth.template_keys(seed, tids)
    q, _ = synth.gaussian_rows(seed, synth.S_QUERY, 0, d, "bf16", row_ids=tids)
    return keys, q


@pytest.mark.parametrize("n_distinct", [1, 31, 32, 33, 64, 65, 96, 97, 128, 129, 161, 200])
def test_bf16_query_blocks(n_distinct):
    d, N, k = 256, 3000, 10
    keys, q = _requests(n_distinct, d)
    c, _ = synth.gaussian_rows(5, synth.S_CORPUS, N, d, "bf16")
    note(f"bf16 n_u={n_distinct}")
    m = run_merge(keys, q, c, k)
    ref = check_dedup(m, keys)
    assert ref["n_unique"] == n_distinct
    check_unique_topk(m, ref, q, c, k)
    check_delivery(m, keys.shape[0])


@pytest.mark.parametrize("n_distinct,k", [(20, 10), (50, 40), (70, 10), (100, 40)])
def test_fp8_query_blocks(n_distinct, k):
    d, N = 128, 2500
    keys, q = _requests(n_distinct, d)
    c, sc = synth.gaussian_rows(6, synth.S_CORPUS, N, d, "fp8")
    note(f"fp8 n_u={n_distinct} k={k}")
    m = run_merge(keys, q, c, k, scale=sc)
    ref = check_dedup(m, keys)
    check_unique_topk(m, ref, q, c, k, scale=sc)
    check_delivery(m, keys.shape[0])


@pytest.mark.parametrize("n_distinct", [10, 45, 80])
def test_bf16_global_lists_query_blocks(n_distinct):
    d, N, k = 128, 4000, 64
    keys, q = _requests(n_distinct, d)
    c, _ = synth.gaussian_rows(7, synth.S_CORPUS, N, d, "bf16")
    m = run_merge(keys, q, c, k)
    ref = check_dedup(m, keys)
    check_unique_topk(m, ref, q, c, k)
