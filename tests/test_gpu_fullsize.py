"""Parity at the full workload sizes, in the launch configuration the
benchmark times (whole path on one stream, distinct count kept on the
device, corpus in the tiled layout).  Dedup, gathers and delivery are checked bit-exactly in full; the
exact top-k is checked for distinct queries spread over every block of 128
consecutive distinct queries (all of them on the 1M-row workload), and for a
seeded sample of requests against an independent, unmerged retrieval of each
request's own query row (each check is an oracle pass over the whole
corpus)."""
import numpy as np
import pytest

import synth
from gpu_harness import (check_dedup, check_delivery, check_requests_vs_oracle,
                         check_unique_topk, note, run_merge)

pytestmark = pytest.mark.gpu

_RUNS = {}


def _run(name):
    """The workload, the GPU result of the whole path and the oracle's dedup,
    computed once per workload for the tests of this module."""
    if name not in _RUNS:
        _RUNS.clear()   # one workload's corpus held at a time
        note(f"{name}: generating")
        w = synth.make(name)
        note(f"{name}: R={w.R} N={w.n_corpus} d={w.dim} k={w.k} corpus={w.corpus.dtype}")
        m = run_merge(w.keys, w.q_req, w.corpus, w.k, scale=w.scale, tiled=True)
        ref = check_dedup(m, w.keys)
        note(f"{name}: dedup exact, n_u={ref['n_unique']}")
        check_delivery(m, w.R)
        _RUNS[name] = (w, m, ref)
    return _RUNS[name]


def spread_sample(nu, per_block, block=128, seed=7):
    """Distinct-query positions: `per_block` seeded positions in every block of
    `block` consecutive distinct queries (fewer in a short last block), plus
    the first and the last."""
    rng = np.random.default_rng(seed)
    picks = [0, nu - 1]
    for b0 in range(0, nu, block):
        n = min(block, nu - b0)
        picks.extend((b0 + rng.choice(n, size=min(per_block, n), replace=False)).tolist())
    return np.unique(np.array(picks, dtype=np.int64))


def _queries(name, per_block):
    w, m, ref = _run(name)
    nu = ref["n_unique"]
    sel = spread_sample(nu, per_block)
    assert len(sel) >= min(nu, 64)
    check_unique_topk(m, ref, w.q_req, w.corpus, w.k, scale=w.scale, sel=sel)
    note(f"{name}: top-k of {len(sel)} of {nu} distinct queries accepted")


def _requests(name, n_req):
    w, m, ref = _run(name)
    rng = np.random.default_rng(11)
    reqs = np.sort(rng.choice(w.R, size=n_req, replace=False))
    check_requests_vs_oracle(m, ref, reqs, w.q_req, w.corpus, w.k, scale=w.scale)
    note(f"{name}: {n_req} requests match independent retrieval")


def test_spread_sample_covers_every_block():
    sel = spread_sample(9995, 1)
    assert sel[0] == 0 and sel[-1] == 9994
    assert set((sel // 128).tolist()) == set(range(79))
    sel = spread_sample(2197, 4)
    assert len(sel) >= 64 and set((sel // 128).tolist()) == set(range(18))


def test_ridge1m_full_size_all_queries():
    # every distinct query of the window (329)
    _queries("ridge1m", 128)


def test_ridge1m_full_size_requests():
    _requests("ridge1m", 64)


@pytest.mark.timeout(900)
def test_mfma4m_full_size_queries():
    # one distinct query in every block of 128 (79 blocks) + the first and last
    _queries("mfma4m", 1)


@pytest.mark.timeout(900)
def test_mfma4m_full_size_requests():
    _requests("mfma4m", 32)


@pytest.mark.timeout(900)
def test_fp8_20m_full_size_queries():
    # four distinct queries in every block of 128 (18 blocks) + the first and last
    _queries("fp8_20m", 4)


@pytest.mark.timeout(900)
def test_fp8_20m_full_size_requests():
    _requests("fp8_20m", 32)
