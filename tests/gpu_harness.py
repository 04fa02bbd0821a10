"""Helpers shared by the GPU parity tests.

Inputs always come from the seeded generator; expected values always come
from the oracle.  GPU outputs are only ever the thing being checked."""
from __future__ import annotations

import os
import sys
import time

import numpy as np
import torch

import oracle
from oracle import accept


def device():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test selected but no GPU is visible")
    return torch.device("cuda:0")


def note(msg: str):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def to_dev(a: np.ndarray, dev=None) -> torch.Tensor:
    """numpy array (generator storage encodings) -> device tensor."""
    dev = dev or device()
    if a.dtype == np.uint16:        # bf16 bit patterns
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def enc_code(a: np.ndarray) -> int:
    import paper_2607_22578_amd as hs
    return {np.dtype(np.float32): hs.HS_F32, np.dtype(np.uint16): hs.HS_BF16,
            np.dtype(np.uint8): hs.HS_FP8_E4M3}[a.dtype]


def run_merge(keys, q_req, corpus, k, scale=None, n_unique_mode="device", max_unique=0,
              tiled=False):
    """Run the whole path on the GPU; returns the MergedRetrieval object
    (outputs still on the device) after a synchronisation.  tiled: score the
    tiled copy of the corpus (made on the device from the row-major one)."""
    import paper_2607_22578_amd as hs
    dev = device()
    R, d = q_req.shape
    N = corpus.shape[0]
    m = hs.MergedRetrieval(R, d, N, k, enc_code(q_req), enc_code(corpus), device=dev,
                           max_unique=max_unique, tiled_corpus=tiled)
    kd, qd, cd = to_dev(keys), to_dev(q_req), to_dev(corpus)
    sd = to_dev(scale) if scale is not None else None
    st = torch.cuda.current_stream(dev)
    if tiled:
        cd = m.tile_corpus(cd, st)
    if n_unique_mode == "host":
        nu = m.dedup(kd, st, host_count=True)
        m.gather_queries(qd, st)
        m.score_partial(cd, sd, nu, st)
        m.topk_merge(nu, st)
        m.deliver(st)
    else:
        m.run(kd, qd, cd, sd, stream=st)
    torch.cuda.synchronize(dev)
    m._inputs = (kd, qd, cd, sd)   # keep alive until the caller is done
    return m


def check_dedup(m, keys):
    ref = oracle.dedup(keys)
    nu = int(m.n_unique.item())
    assert nu == ref["n_unique"], (nu, ref["n_unique"])
    R = keys.shape[0]
    np.testing.assert_array_equal(m.unique_keys[:nu].cpu().numpy(), ref["unique_keys"])
    np.testing.assert_array_equal(m.first_index[:nu].cpu().numpy(), ref["first_index"])
    np.testing.assert_array_equal(m.counts[:nu].cpu().numpy(), ref["counts"])
    np.testing.assert_array_equal(m.inverse[:R].cpu().numpy(), ref["inverse"])
    return ref


def check_unique_topk(m, ref_dedup, q_req, corpus, k, scale=None, sel=None, threads=None):
    """Acceptance rule on distinct queries `sel` (positions in the distinct
    list; all when None).  Returns the checked positions."""
    nu = ref_dedup["n_unique"]
    if sel is None:
        sel = np.arange(nu)
    sel = np.asarray(sel, dtype=np.int64)
    rows = ref_dedup["first_index"][sel].astype(np.int64)
    N = corpus.shape[0]
    rs, ri = oracle.topk_exact(q_req, corpus, k + 1, scale=scale, q_rows=rows, threads=threads)
    gs = m.topk_score[sel].cpu().numpy()
    gi = m.topk_index[sel].cpu().numpy().astype(np.int64)
    valid = gi >= 0
    qi = np.repeat(rows, k).reshape(len(sel), k)
    ex = np.full(gi.shape, np.nan)
    if valid.any():
        ex[valid] = oracle.score_pairs(q_req, corpus, qi[valid], gi[valid], scale=scale,
                                       threads=threads)
    bad = accept.check_all(gs, gi, rs, ri, ex, N, k, labels=sel.tolist())
    assert not bad, f"{len(bad)} queries violate the acceptance rule, first: {bad[:3]}"
    return sel


def check_delivery(m, R):
    """out[i] == topk[inverse[i]] bit-exactly for every request."""
    inv = m.inverse[:R].long()
    np.testing.assert_array_equal(m.out_index[:R].cpu().numpy(),
                                  m.topk_index[inv].cpu().numpy())
    a = m.out_score[:R].cpu().numpy().view(np.uint32)
    b = m.topk_score[inv].cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(a, b)


def check_requests_vs_oracle(m, ref_dedup, sel_requests, q_req, corpus, k, scale=None):
    """Per-request outputs of selected requests: same acceptance rule against
    an independent (unmerged) retrieval of the request's own query row."""
    sel_requests = np.asarray(sel_requests, dtype=np.int64)
    N = corpus.shape[0]
    rs, ri = oracle.topk_exact(q_req, corpus, k + 1, scale=scale, q_rows=sel_requests)
    gs = m.out_score[sel_requests].cpu().numpy()
    gi = m.out_index[sel_requests].cpu().numpy().astype(np.int64)
    valid = gi >= 0
    qi = np.repeat(sel_requests, k).reshape(len(sel_requests), k)
    ex = np.full(gi.shape, np.nan)
    if valid.any():
        ex[valid] = oracle.score_pairs(q_req, corpus, qi[valid], gi[valid], scale=scale)
    bad = accept.check_all(gs, gi, rs, ri, ex, N, k, labels=sel_requests.tolist())
    assert not bad, f"{len(bad)} requests violate the acceptance rule, first: {bad[:3]}"
