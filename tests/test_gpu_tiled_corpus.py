"""The tiled corpus layout (hs_tile_corpus, HS_FLAG_TILED_CORPUS): the tiled
copy byte for byte against a numpy re-layout written here from the layout's
definition in hs_merge.h, and the score step on it against the row-major
corpus (bit-identical outputs: the kernel's LDS contents are the same) and
against the oracle, on ragged corpora, partial last K stages, the largest
dimension (d = 16,384), k-lists in LDS
and in global memory, several query tiles and the no-allocation entry point."""
import numpy as np
import pytest
import torch

import paper_2607_22578_amd as hs
import synth
from gpu_harness import (check_dedup, check_delivery, check_unique_topk, device, enc_code, note,
                         run_merge, to_dev)

pytestmark = pytest.mark.gpu


def _stream(n_corpus: int, d: int, enc: str, workload: str = "ridge1m"):
    w = synth.make(workload, n_corpus=1, with_corpus=False)
    q, _ = synth.gaussian_rows(w.seed, synth.S_QUERY, 0, d, "bf16", row_ids=w.template_ids)
    c, sc = synth.gaussian_rows(w.seed, synth.S_CORPUS, n_corpus, d, enc)
    return w, q, c, sc


def _tiled_numpy(c: np.ndarray) -> np.ndarray:
    """Blocks of 384 rows x 64 columns, block (t, s) at (t * S + s), rows in
    order, the 16-byte pieces of row r permuted: slot x holds piece
    x XOR ((r // (16 / P)) mod P), P = pieces per 64-column row segment;
    zeros past N and d."""
    N, d = c.shape
    esz = c.dtype.itemsize
    P = 64 * esz // 16
    T, S = -(-N // 384), -(-d // 64)
    pad = np.zeros((T * 384, S * 64 * esz), np.uint8)
    pad[:N, :d * esz] = np.ascontiguousarray(c).view(np.uint8).reshape(N, d * esz)
    blocks = pad.reshape(T, 384, S, P, 16).transpose(0, 2, 1, 3, 4)   # t, s, r, piece, byte
    r = np.arange(384)[:, None]
    perm = np.arange(P)[None, :] ^ ((r // (16 // P)) % P)
    return blocks[:, :, r, perm].reshape(-1)


@pytest.mark.parametrize("enc,N,d", [("bf16", 1000, 200), ("bf16", 384, 64), ("bf16", 385, 776),
                                     ("fp8", 1000, 208), ("fp8", 7, 16), ("fp8", 800, 1024)])
def test_tiled_copy_bytes(enc, N, d):
    w, q, c, _ = _stream(N, d, enc)
    note(f"tile {enc} N={N} d={d}")
    p = hs.hs_merge_plan(64, d, N, 10, hs.HS_BF16, enc_code(c), flags=hs.HS_FLAG_TILED_CORPUS)
    m_bytes = hs.hs_corpus_tiled_bytes(p)
    dev = device()
    cd = to_dev(c, dev)
    # a guard past the end must stay untouched
    out = torch.full((m_bytes + 4096,), 0xA5, dtype=torch.uint8, device=dev)
    hs.hs_tile_corpus(p, cd, out, m_bytes)
    torch.cuda.synchronize(dev)
    got = out.cpu().numpy()
    np.testing.assert_array_equal(got[:m_bytes], _tiled_numpy(c))
    assert (got[m_bytes:] == 0xA5).all()


def _same_outputs(a, b, R):
    nu = int(a.n_unique.item())
    assert nu == int(b.n_unique.item())
    for x, y in ((a.topk_score[:nu], b.topk_score[:nu]), (a.out_score[:R], b.out_score[:R])):
        np.testing.assert_array_equal(x.cpu().numpy().view(np.uint32),
                                      y.cpu().numpy().view(np.uint32))
    for x, y in ((a.topk_index[:nu], b.topk_index[:nu]), (a.out_index[:R], b.out_index[:R])):
        np.testing.assert_array_equal(x.cpu().numpy(), y.cpu().numpy())


@pytest.mark.parametrize("enc,N,d,k", [
    ("bf16", 2000, 200, 10),      # partial last stage, ragged tile
    ("bf16", 6000, 768, 64),      # k-lists in global memory
    ("bf16", 20011, 128, 100),    # seed sample over several tiles
    ("fp8", 2500, 784, 10),
    ("fp8", 9000, 512, 100),
])
def test_tiled_matches_rows_and_oracle(enc, N, d, k):
    w, q, c, sc = _stream(N, d, enc)
    note(f"tiled vs rows {enc} N={N} d={d} k={k}")
    rows = run_merge(w.keys, q, c, k, scale=sc)
    tiled = run_merge(w.keys, q, c, k, scale=sc, tiled=True)
    _same_outputs(rows, tiled, w.R)
    ref = check_dedup(tiled, w.keys)
    check_unique_topk(tiled, ref, q, c, k, scale=sc)
    check_delivery(tiled, w.R)


def test_tiled_several_query_tiles():
    # 4,096 requests with more than 128 distinct queries: several query tiles
    w, q, c, sc = _stream(30000, 256, "bf16", workload="mfma4m")
    keys, q = w.keys[:4096], q[:4096]
    note("tiled several query tiles")
    rows = run_merge(keys, q, c, 32)
    tiled = run_merge(keys, q, c, 32, tiled=True)
    assert int(tiled.n_unique.item()) > 256
    _same_outputs(rows, tiled, 4096)
    ref = check_dedup(tiled, keys)
    sel = np.random.default_rng(3).choice(ref["n_unique"], size=64, replace=False)
    check_unique_topk(tiled, ref, q, c, 32, sel=sel)


def test_tiled_noalloc_and_host_count():
    w, q, c, _ = _stream(5000, 384, "bf16")
    note("tiled noalloc")
    a = run_merge(w.keys, q, c, 10, tiled=True, n_unique_mode="host")
    b = run_merge(w.keys, q, c, 10, tiled=False)
    _same_outputs(a, b, w.R)
    # the no-allocation entry point on the same tiled copy
    nu = int(a.n_unique.item())
    dev = device()
    ts = torch.empty((nu, 10), dtype=torch.float32, device=dev)
    ti = torch.empty((nu, 10), dtype=torch.int32, device=dev)
    hs.hs_score_topk_noalloc(a.plan, a.q_unique, nu, None, a._inputs[2], None, ts, ti)
    torch.cuda.synchronize(dev)
    np.testing.assert_array_equal(ts.cpu().numpy().view(np.uint32),
                                  a.topk_score[:nu].cpu().numpy().view(np.uint32))
    np.testing.assert_array_equal(ti.cpu().numpy(), a.topk_index[:nu].cpu().numpy())


@pytest.mark.parametrize("enc", ["bf16", "fp8"])
def test_max_dimension_both_layouts(enc):
    # d = 16,384 (the largest the plan accepts): 256 stages per tile, 12 MiB
    # bf16 tiles, over a ragged corpus of four tiles
    w, q, c, sc = _stream(1500, 16384, enc, workload="tiny")
    note(f"max dimension {enc}")
    rows = run_merge(w.keys, q, c, w.k, scale=sc)
    tiled = run_merge(w.keys, q, c, w.k, scale=sc, tiled=True)
    _same_outputs(rows, tiled, w.R)
    ref = check_dedup(tiled, w.keys)
    check_unique_topk(tiled, ref, q, c, w.k, scale=sc)
    check_delivery(tiled, w.R)
