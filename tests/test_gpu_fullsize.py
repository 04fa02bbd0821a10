"""Parity at the full workload sizes, in the launch configuration the
benchmark times (whole path on one stream, distinct count kept on the
device).  Dedup, gathers and delivery are checked bit-exactly in full; the
exact top-k is checked for a seeded sample of distinct queries and requests
(each one an oracle pass over the whole corpus)."""
import numpy as np
import pytest

import synth
from gpu_harness import (check_dedup, check_delivery, check_requests_vs_oracle,
                         check_unique_topk, note, run_merge)

pytestmark = pytest.mark.gpu


def _sampled_check(name, n_sample_unique, n_sample_req):
    note(f"{name}: generating")
    w = synth.make(name)
    note(f"{name}: R={w.R} N={w.n_corpus} d={w.dim} k={w.k} corpus={w.corpus.dtype}")
    m = run_merge(w.keys, w.q_req, w.corpus, w.k, scale=w.scale)
    ref = check_dedup(m, w.keys)
    nu = ref["n_unique"]
    note(f"{name}: dedup exact, n_u={nu}")
    check_delivery(m, w.R)
    rng = np.random.default_rng(7)
    # always include the first and last distinct query (first and last query
    # tile / group) plus a seeded sample in between
    sel = np.unique(np.concatenate([[0, nu - 1],
                                    rng.choice(nu, size=n_sample_unique, replace=False)]))
    check_unique_topk(m, ref, w.q_req, w.corpus, w.k, scale=w.scale, sel=sel)
    note(f"{name}: top-k of {len(sel)} distinct queries accepted")
    reqs = rng.choice(w.R, size=n_sample_req, replace=False)
    check_requests_vs_oracle(m, ref, reqs, w.q_req, w.corpus, w.k, scale=w.scale)
    note(f"{name}: {n_sample_req} requests match independent retrieval")


def test_ridge1m_full_size():
    _sampled_check("ridge1m", 14, 8)


def test_mfma4m_full_size():
    _sampled_check("mfma4m", 6, 4)


def test_fp8_20m_full_size():
    _sampled_check("fp8_20m", 4, 3)
