"""The C ABI: the library loads, exports every declared symbol, and rejects bad
arguments on the host before any HIP call (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2607_22578_amd as hs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "hs_merge.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(hs_[a-z_]+)\s*\(", txt)))


def test_exports_every_declared_symbol():
    decl = _declared()
    assert set(decl) == set(hs.EXPORTS), decl
    lib = ctypes.CDLL(hs.LIB_PATH)
    for name in decl:
        assert hasattr(lib, name), name


def test_abi_version_and_status_strings():
    assert hs.hs_abi_version() == hs.ABI_VERSION == 3
    assert hs.hs_status_string(hs.HS_OK) == "HS_OK"
    assert hs.hs_status_string(hs.HS_ERR_WORKSPACE) == "HS_ERR_WORKSPACE"
    assert hs.hs_status_string(99) == "HS_ERR_UNKNOWN"


GOOD = dict(n_requests=2048, dim=768, n_corpus=1_000_000, k=10, query_dtype=hs.HS_BF16,
            corpus_dtype=hs.HS_BF16)


def test_plan_ok_and_workspace():
    p = hs.hs_merge_plan(**GOOD)
    assert p.workspace_bytes > 0
    p2 = hs.hs_merge_plan(**dict(GOOD, n_requests=262_144, k=10))
    assert p2.workspace_bytes >= 262_144 * 24   # radix dedup buffers
    p3 = hs.hs_merge_plan(**dict(GOOD, n_requests=0))
    assert p3.workspace_bytes >= 0


@pytest.mark.parametrize("bad,code", [
    (dict(k=0), hs.HS_ERR_INVALID_ARG),
    (dict(k=1025), hs.HS_ERR_INVALID_ARG),
    (dict(dim=0), hs.HS_ERR_INVALID_ARG),
    (dict(dim=20000), hs.HS_ERR_INVALID_ARG),
    (dict(dim=764), hs.HS_ERR_UNSUPPORTED),                      # bf16 needs d % 8
    (dict(dim=776, corpus_dtype=hs.HS_FP8_E4M3), hs.HS_ERR_UNSUPPORTED),  # fp8 needs d % 16
    (dict(n_requests=-1), hs.HS_ERR_INVALID_ARG),
    (dict(n_requests=2 ** 31), hs.HS_ERR_INVALID_ARG),
    (dict(n_requests=2 ** 30 + 1), hs.HS_ERR_INVALID_ARG),
    (dict(n_corpus=-5), hs.HS_ERR_INVALID_ARG),
    (dict(n_corpus=2 ** 31), hs.HS_ERR_INVALID_ARG),
    (dict(query_dtype=7), hs.HS_ERR_UNSUPPORTED),
    (dict(query_dtype=hs.HS_F32), hs.HS_ERR_UNSUPPORTED),         # f32 queries + bf16 corpus
    (dict(corpus_dtype=hs.HS_F32), hs.HS_ERR_UNSUPPORTED),        # bf16 queries + f32 corpus
    (dict(max_unique=5000), hs.HS_ERR_INVALID_ARG),
    (dict(flags=2), hs.HS_ERR_INVALID_ARG),                       # unknown flag bit
    (dict(flags=-1), hs.HS_ERR_INVALID_ARG),
    (dict(flags=hs.HS_FLAG_TILED_CORPUS, query_dtype=hs.HS_F32, corpus_dtype=hs.HS_F32),
     hs.HS_ERR_UNSUPPORTED),                                      # tiled: BF16/FP8 only
])
def test_plan_rejects(bad, code):
    with pytest.raises(hs.HsError) as e:
        hs.hs_merge_plan(**dict(GOOD, **bad))
    assert e.value.status == code
    assert hs.hs_last_error()


def test_workflow_offsets_uniform_and_csr():
    # NULL offsets: W equal workflows of R / W requests
    p = hs.hs_merge_plan(**GOOD, n_workflows=64)
    assert [hs.hs_workflow_rows(p, w) for w in (0, 1, 63)] == [(0, 32), (32, 32), (2016, 32)]
    # an explicit CSR (empty workflows allowed), copied by the plan
    off = [0, 5, 5, 1000, 2048]
    p = hs.hs_merge_plan(**GOOD, n_workflows=4, workflow_offsets=off)
    off[1] = 999   # the caller's array is not kept
    assert [hs.hs_workflow_rows(p, w) for w in range(4)] == [(0, 5), (5, 0), (5, 995),
                                                             (1000, 1048)]
    for w in (-1, 4):
        with pytest.raises(hs.HsError) as e:
            hs.hs_workflow_rows(p, w)
        assert e.value.status == hs.HS_ERR_INVALID_ARG
    # one workflow holding the whole (possibly empty) window
    assert hs.hs_workflow_rows(hs.hs_merge_plan(**dict(GOOD, n_requests=0)), 0) == (0, 0)


@pytest.mark.parametrize("W,off", [
    (0, None),                      # at least one workflow
    (-3, None),
    (2 ** 30 + 1, None),
    (3, None),                      # 3 does not divide 2048 without offsets
    (3, [1, 5, 9, 2048]),           # must start at 0
    (3, [0, 5, 9, 2047]),           # must end at R
    (3, [0, 9, 5, 2048]),           # decreasing
    (2, [0, 2049, 2048]),           # decreasing at the end
])
def test_workflow_offsets_rejected(W, off):
    with pytest.raises(hs.HsError) as e:
        hs.hs_merge_plan(**GOOD, n_workflows=W, workflow_offsets=off)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    assert "workflow" in hs.hs_last_error()


FAKE = 0x10000000   # never dereferenced: validation fails first


def _tiled_size(N, d, esz):
    # 384-row x 64-column blocks, rows and columns padded with zeros
    return -(-N // 384) * 384 * (-(-d // 64) * 64) * esz


@pytest.mark.parametrize("N,d,cdt,esz", [
    (1_000_000, 768, hs.HS_BF16, 2), (384, 64, hs.HS_BF16, 2), (385, 72, hs.HS_BF16, 2),
    (1000, 208, hs.HS_FP8_E4M3, 1), (20_000_000, 512, hs.HS_FP8_E4M3, 1), (0, 128, hs.HS_BF16, 2),
])
def test_corpus_tiled_bytes(N, d, cdt, esz):
    for flags in (0, hs.HS_FLAG_TILED_CORPUS):
        p = hs.hs_merge_plan(**dict(GOOD, n_corpus=N, dim=d, corpus_dtype=cdt, flags=flags))
        assert hs.hs_corpus_tiled_bytes(p) == _tiled_size(N, d, esz)


def test_tile_corpus_validation():
    f32 = hs.hs_merge_plan(**dict(GOOD, query_dtype=hs.HS_F32, corpus_dtype=hs.HS_F32))
    for call in (lambda: hs.hs_corpus_tiled_bytes(f32),
                 lambda: hs.hs_tile_corpus(f32, FAKE, FAKE, 1 << 40)):
        with pytest.raises(hs.HsError) as e:
            call()
        assert e.value.status == hs.HS_ERR_UNSUPPORTED
    p = hs.hs_merge_plan(**GOOD)
    need = hs.hs_corpus_tiled_bytes(p)
    cases = [
        ((None, FAKE, need), hs.HS_ERR_INVALID_ARG),            # null corpus
        ((FAKE, None, need), hs.HS_ERR_INVALID_ARG),            # null tiled buffer
        ((FAKE, FAKE + (1 << 33), need - 16), hs.HS_ERR_INVALID_ARG),   # buffer too small
        ((FAKE + 8, FAKE + (1 << 33), need), hs.HS_ERR_ALIGNMENT),
        ((FAKE, FAKE + (1 << 33) + 4, need), hs.HS_ERR_ALIGNMENT),
        ((FAKE, FAKE + 4096, need), hs.HS_ERR_INVALID_ARG),     # overlaps the corpus
        ((FAKE + 4096, FAKE, need), hs.HS_ERR_INVALID_ARG),
    ]
    for (c, t, nb), code in cases:
        with pytest.raises(hs.HsError) as e:
            hs.hs_tile_corpus(p, c, t, nb)
        assert e.value.status == code, (c, t, nb)
    # an empty corpus: nothing to write, nothing enqueued
    p0 = hs.hs_merge_plan(**dict(GOOD, n_corpus=0))
    assert hs.hs_corpus_tiled_bytes(p0) == 0
    hs.hs_tile_corpus(p0, None, None, 0)


def test_deliver_validation():
    p = hs.hs_merge_plan(**GOOD)
    hs.hs_deliver(p, FAKE, FAKE, 0, FAKE, FAKE, FAKE)   # no rows: nothing enqueued
    with pytest.raises(hs.HsError) as e:
        hs.hs_deliver(p, FAKE, FAKE, -1, FAKE, FAKE, FAKE)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:
        hs.hs_deliver(p, FAKE, None, 10, FAKE, FAKE, FAKE)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:
        hs.hs_deliver(p, FAKE, FAKE, 10, FAKE + 2, FAKE, FAKE)
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    # a null plan, through the C entry point itself
    assert hs._lib.hs_deliver(None, FAKE, FAKE, 10, FAKE, FAKE, FAKE, None) == \
        hs.HS_ERR_INVALID_ARG


def test_dedup_validation():
    p = hs.hs_merge_plan(**dict(GOOD, n_requests=100_000))
    with pytest.raises(hs.HsError) as e:   # no workspace
        hs.hs_dedup(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0)
    assert e.value.status == hs.HS_ERR_WORKSPACE
    with pytest.raises(hs.HsError) as e:   # workspace too small
        hs.hs_dedup(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1000)
    assert e.value.status == hs.HS_ERR_WORKSPACE
    with pytest.raises(hs.HsError) as e:   # misaligned keys
        hs.hs_dedup(p, FAKE + 4, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, p.workspace_bytes)
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    with pytest.raises(hs.HsError) as e:   # null output
        hs.hs_dedup(p, FAKE, None, FAKE, FAKE, FAKE, FAKE, None, FAKE, p.workspace_bytes)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:   # misaligned workspace
        hs.hs_dedup(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE + 16, p.workspace_bytes)
    assert e.value.status == hs.HS_ERR_ALIGNMENT


def test_score_validation():
    p = hs.hs_merge_plan(**GOOD)
    ws = p.workspace_bytes
    with pytest.raises(hs.HsError) as e:   # n_unique beyond the plan
        hs.hs_score_topk(p, FAKE, 4096, None, FAKE, None, FAKE, FAKE, FAKE, ws)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:   # -1 without device count
        hs.hs_score_topk(p, FAKE, -1, None, FAKE, None, FAKE, FAKE, FAKE, ws)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:   # misaligned corpus
        hs.hs_score_topk(p, FAKE, 10, None, FAKE + 2, None, FAKE, FAKE, FAKE, ws)
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    with pytest.raises(hs.HsError) as e:   # workspace too small
        hs.hs_score_partial(p, FAKE, 10, None, FAKE, None, FAKE, ws - 1)
    assert e.value.status == hs.HS_ERR_WORKSPACE
    with pytest.raises(hs.HsError) as e:
        hs.hs_topk_merge(p, 10, None, None, FAKE, FAKE, ws)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    p8 = hs.hs_merge_plan(**dict(GOOD, corpus_dtype=hs.HS_FP8_E4M3))
    with pytest.raises(hs.HsError) as e:   # fp8 without row scale
        hs.hs_score_topk(p8, FAKE, 10, None, FAKE, None, FAKE, FAKE, FAKE, p8.workspace_bytes)
    assert e.value.status == hs.HS_ERR_INVALID_ARG


def test_scatter_validation():
    with pytest.raises(hs.HsError) as e:
        hs.hs_scatter(FAKE, 10, 6, FAKE, 0, 5, None, FAKE)      # row_bytes % 4
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:
        hs.hs_scatter(FAKE, 10, 8, FAKE, 2, 5, None, FAKE)      # bad index flag
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:
        hs.hs_scatter(FAKE, 10, 8, FAKE + 4, 1, 5, None, FAKE)  # misaligned i64 index
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    with pytest.raises(hs.HsError) as e:
        hs.hs_scatter(None, 10, 8, FAKE, 0, 5, None, FAKE)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    # empty work is a no-op that never touches the device
    hs.hs_scatter(FAKE, 10, 8, FAKE, 0, 0, None, FAKE)


def test_cache_validation():
    p = hs.hs_merge_plan(**GOOD)
    assert hs.hs_cache_bytes(p, 1) >= 8 + 4 + 4 + 2 * 10 * 4
    b = hs.hs_cache_bytes(p, 4096)
    assert b >= 4096 * (16 + 80) and b % 256 == 0
    for bad in (0, 3, 6000, -4, 2 ** 31):
        with pytest.raises(hs.HsError) as e:
            hs.hs_cache_bytes(p, bad)
        assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:        # store buffer too small
        hs.hs_cache_reset(p, FAKE, 4096, cache_bytes=b - 1)
    assert e.value.status == hs.HS_ERR_WORKSPACE
    with pytest.raises(hs.HsError) as e:        # misaligned store
        hs.hs_cache_reset(p, FAKE + 16, 4096, cache_bytes=b)
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    with pytest.raises(hs.HsError) as e:        # capacity not a power of two
        hs.hs_cache_reset(p, FAKE, 4095, cache_bytes=b)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:        # n_unique beyond the plan
        hs.hs_cache_lookup(p, FAKE, 4096, FAKE, FAKE, 4096, None, FAKE, FAKE, FAKE, FAKE, FAKE,
                           cache_bytes=b)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:        # null miss count
        hs.hs_cache_lookup(p, FAKE, 4096, FAKE, FAKE, 10, None, FAKE, FAKE, FAKE, FAKE, None,
                           cache_bytes=b)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:        # misaligned keys
        hs.hs_cache_lookup(p, FAKE, 4096, FAKE + 4, FAKE, 10, None, FAKE, FAKE, FAKE, FAKE,
                           FAKE, cache_bytes=b)
    assert e.value.status == hs.HS_ERR_ALIGNMENT
    with pytest.raises(hs.HsError) as e:        # -1 without a device count
        hs.hs_cache_insert(p, FAKE, 4096, FAKE, FAKE, -1, None, FAKE, FAKE, cache_bytes=b)
    assert e.value.status == hs.HS_ERR_INVALID_ARG
    with pytest.raises(hs.HsError) as e:
        hs.hs_cache_insert(p, FAKE, 4096, FAKE, None, 10, None, FAKE, FAKE, cache_bytes=b)
    assert e.value.status == hs.HS_ERR_INVALID_ARG


def test_signature_validation():
    def call(n=10, first=0, count=10, flags=0, digest=FAKE, keys=FAKE, **kw):
        base = dict(op_type=FAKE, text=FAKE, text_off=FAKE, text_bytes=100)
        base.update(kw)
        hs.hs_signature(base.pop("op_type"), n, first, count, digest, keys, flags=flags,
                        **base)

    for bad in (dict(n=-1), dict(n=2 ** 27 + 1), dict(first=-1), dict(count=11),
                dict(first=5, count=6), dict(flags=2), dict(text_bytes=2 ** 32),
                dict(op_type=None), dict(digest=None), dict(text=None),
                dict(pred_off=FAKE, pred_idx=None, pred_count=3),
                dict(pred_off=FAKE, pred_idx=FAKE, pred_count=2 ** 31)):
        with pytest.raises(hs.HsError) as e:
            call(**bad)
        assert e.value.status == hs.HS_ERR_INVALID_ARG, bad
    for bad in (dict(digest=FAKE + 8), dict(keys=FAKE + 4), dict(op_type=FAKE + 2),
                dict(text_off=FAKE + 4)):
        with pytest.raises(hs.HsError) as e:
            call(**bad)
        assert e.value.status == hs.HS_ERR_ALIGNMENT, bad
    call(count=0, first=10)   # empty range: nothing is enqueued


def test_priority_validation():
    p = hs.hs_merge_plan(**GOOD)
    ws = p.workspace_bytes
    args = [FAKE, FAKE, 10, None, FAKE, FAKE, None, 1.0, 1.0, 0.0, 1e-3, FAKE, FAKE, FAKE, FAKE]
    hs.hs_priority(p, *args[:2], 0, None, *args[4:], ws_bytes=ws)   # n_u = 0: no-op
    for i, bad, code in [(2, 4096, hs.HS_ERR_INVALID_ARG),          # beyond the plan
                         (2, -1, hs.HS_ERR_INVALID_ARG),            # -1 without device count
                         (10, 0.0, hs.HS_ERR_INVALID_ARG),          # eps must be > 0
                         (7, float("nan"), hs.HS_ERR_INVALID_ARG),  # alpha finite
                         (0, None, hs.HS_ERR_INVALID_ARG),
                         (13, None, hs.HS_ERR_INVALID_ARG),         # order
                         (11, FAKE + 4, hs.HS_ERR_ALIGNMENT),       # fp64 output
                         (14, FAKE + 64, hs.HS_ERR_ALIGNMENT)]:     # workspace
        a = list(args)
        a[i] = bad
        with pytest.raises(hs.HsError) as e:
            hs.hs_priority(p, *a, ws_bytes=ws)
        assert e.value.status == code, (i, bad)
    with pytest.raises(hs.HsError) as e:
        hs.hs_priority(p, *args, ws_bytes=16)
    assert e.value.status == hs.HS_ERR_WORKSPACE


def test_noalloc_validation():
    # rejected on the host, before the scratch array is touched
    big = hs.hs_merge_plan(32768, 1024, 4_000_000, 32, hs.HS_BF16, hs.HS_BF16)
    with pytest.raises(hs.HsError) as e:
        hs.hs_score_topk_noalloc(big, FAKE, 10, None, FAKE, None, FAKE, FAKE)
    assert e.value.status == hs.HS_ERR_WORKSPACE and "scratch" in hs.hs_last_error()
    p = hs.hs_merge_plan(**GOOD)
    for args, code in [((FAKE, 4096, None, FAKE, None, FAKE, FAKE), hs.HS_ERR_INVALID_ARG),
                       ((FAKE, -1, None, FAKE, None, FAKE, FAKE), hs.HS_ERR_INVALID_ARG),
                       ((FAKE, 10, None, FAKE + 2, None, FAKE, FAKE), hs.HS_ERR_ALIGNMENT),
                       ((FAKE, 10, None, FAKE, None, None, FAKE), hs.HS_ERR_INVALID_ARG)]:
        with pytest.raises(hs.HsError) as e:
            hs.hs_score_topk_noalloc(p, *args)
        assert e.value.status == code, args
