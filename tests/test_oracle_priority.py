"""Pins of the oracle's fused-node priorities (oracle/priority.py) against
facts fixed outside it: a hand-worked example (tests/golden), the closed form
of Eq. 3 for equal contributions, the special cases of Eq. 7 that reduce to
shortest-remaining-time-first, to ordering by reuse gain and to heavy nodes
first, the truncation and clamping rules, and exactness against math.fsum."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import priority as pr

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "priority_worked.json")


def test_hand_worked_example():
    d = json.load(open(GOLDEN))
    phi_f, pi, order = pr.priorities(np.array(d["inverse"]), np.array(d["first_index"]),
                                     np.array(d["phi"], np.float32),
                                     np.array(d["s_hat"], np.float32),
                                     np.array(d["heavy"], np.uint8), d["alpha"], d["gamma"],
                                     d["delta"], d["eps"])
    assert phi_f.tolist() == d["phi_fused"]
    assert pi.tolist() == d["pi"]
    assert order.tolist() == d["order"]


def _groups(rng, R, n_u):
    inv = np.sort(rng.integers(0, n_u, size=R))
    inv[:n_u] = np.arange(n_u)          # every group present
    inv = rng.permutation(inv).astype(np.int32)
    first = np.array([np.nonzero(inv == g)[0][0] for g in range(n_u)], dtype=np.int32)
    return inv, first


def test_equal_contributions_closed_form():
    rng = np.random.default_rng(1)
    inv, first = _groups(rng, 500, 40)
    phi = np.full(500, 1.5, np.float32)
    phi_f, _, _ = pr.priorities(inv, first, phi, np.ones(500, np.float32), None, 0, 1, 0, 1)
    counts = np.bincount(inv, minlength=40)
    assert phi_f.tolist() == (1.5 * counts).tolist()


def test_srtf_special_case():
    rng = np.random.default_rng(2)
    inv, first = _groups(rng, 300, 50)
    s = rng.integers(1, 20, size=300).astype(np.float32)
    _, pi, order = pr.priorities(inv, first, rng.random(300).astype(np.float32), s, None,
                                 1.0, 0.0, 0.0, 0.5)
    # alpha > 0, gamma = delta = 0: shortest remaining time of the survivor first
    expect = sorted(range(50), key=lambda g: (float(s[first[g]]), g))
    assert order.tolist() == expect


def test_reuse_gain_special_case():
    rng = np.random.default_rng(3)
    inv, first = _groups(rng, 400, 30)
    phi = np.full(400, 2.0, np.float32)
    _, _, order = pr.priorities(inv, first, phi, np.ones(400, np.float32), None, 0.0, 1.0,
                                0.0, 1.0)
    counts = np.bincount(inv, minlength=30)
    # equal per-node contributions: the most shared fused node first
    assert order.tolist() == sorted(range(30), key=lambda g: (-counts[g], g))


def test_heavy_first_special_case():
    rng = np.random.default_rng(4)
    inv, first = _groups(rng, 200, 25)
    heavy = (rng.random(200) < 0.3).astype(np.uint8)
    _, _, order = pr.priorities(inv, first, np.ones(200, np.float32), np.ones(200, np.float32),
                                heavy, 0.0, 0.0, 1.0, 1.0)
    y = heavy[first]
    assert order.tolist() == sorted(range(25), key=lambda g: (-int(y[g]), g))


def test_truncation_and_clamping():
    assert pr.phi_units(np.array([2.0 ** -25, 3 * 2.0 ** -24, 1 + 2.0 ** -23], np.float32)) == \
        [0, 3, (1 << 24) + 2]
    top = math.floor(65535.99609375 * 2 ** 24)   # the largest fp32 below 2^16, in units
    assert pr.phi_units(np.array([-1.0, np.nan, 0.0, 1e9, np.inf], np.float32)) == \
        [0, 0, 0, top, top]


def test_exact_sum_matches_fsum():
    rng = np.random.default_rng(5)
    inv, first = _groups(rng, 3000, 7)
    phi = (rng.random(3000) * 100).astype(np.float32)
    phi_f, _, _ = pr.priorities(inv, first, phi, np.ones(3000, np.float32), None, 0, 1, 0, 1)
    for g in range(7):
        trunc = [math.floor(float(x) * 2 ** 24) / 2 ** 24 for x in phi[inv == g]]
        assert phi_f[g] == math.fsum(trunc)


def test_survivor_reading_and_dedup_groups():
    keys = np.array([7, 3, 7, 3, 9], np.int64)
    ref = oracle.dedup(keys)   # groups by ascending key: 3, 7, 9
    s = np.array([8.0, 0.5, 0.25, 4.0, 1.0], np.float32)
    _, pi, _ = pr.priorities(ref["inverse"], ref["first_index"], np.zeros(5, np.float32), s,
                             None, 1.0, 0.0, 0.0, 1.0)
    # group of key 3: first request 1 (S = 0.5); key 7: request 0 (S = 8), not request 2
    assert pi.tolist() == [1 / 1.5, 1 / 9.0, 1 / 2.0]
