"""Pins of the oracle's cross-window result store model (oracle/store.py)
against facts fixed outside it: the multiplier of Fibonacci hashing from the
golden ratio, the real-number form of multiplicative hashing, set semantics
when no two keys share an entry, the one-entry store, and result invariance
(a reused row is the row the same key computes afresh)."""
from decimal import Decimal, getcontext

import numpy as np
import pytest

import oracle
from oracle import store
import synth


def test_multiplier_is_two_pow_64_over_phi():
    getcontext().prec = 60
    phi = (1 + Decimal(5).sqrt()) / 2
    assert store.FIB_MULT == int(Decimal(2) ** 64 / phi)
    assert store.FIB_MULT % 2 == 1   # odd: key -> key * mult mod 2^64 is a bijection


def test_entry_matches_real_number_form():
    # Knuth's multiplicative hashing: entry = floor(C * frac(key / phi)); the
    # integer form agrees except within key / 2^64 of an entry boundary
    getcontext().prec = 60
    inv_phi = 2 / (1 + Decimal(5).sqrt())
    for C in (2, 64, 1024, 1 << 20):
        for key in list(range(1, 600)) + [10 ** 9 + 7, 2 ** 40 + 3]:
            x = Decimal(key) * inv_phi
            frac = x - int(x)
            assert store.entry_of(key, C) == int(frac * C), (key, C)


def test_entry_of_negative_keys_uses_twos_complement():
    C = 1 << 16
    assert store.entry_of(-1, C) == store.entry_of(2 ** 64 - 1, C)
    assert store.entry_of(-(2 ** 63), C) == store.entry_of(2 ** 63, C)
    # -1 * m mod 2^64 = 2^64 - m
    assert store.entry_of(-1, C) == (2 ** 64 - store.FIB_MULT) >> 48


def test_entry_range_and_one_entry_store():
    rng = np.random.default_rng(1)
    keys = rng.integers(-2 ** 63, 2 ** 63 - 1, size=2000, dtype=np.int64)
    for C in (1, 2, 8, 4096):
        e = [store.entry_of(int(k), C) for k in keys]
        assert min(e) >= 0 and max(e) < C
        if C == 1:
            assert set(e) == {0}
    with pytest.raises(ValueError):
        store.entry_of(5, 3)


def _fake_compute(w, miss_keys):
    # a stand-in result that is a function of the key alone
    s = np.array([[float(k % 997), float(k % 13)] for k in miss_keys], dtype=np.float32)
    i = np.array([[int(k % 101), int(k % 7)] for k in miss_keys], dtype=np.int32)
    return s.reshape(-1, 2), i.reshape(-1, 2)


def _windows(n):
    return [w.keys for w in synth.window_stream("ridge1m", n)]


def test_no_sharing_is_set_semantics():
    wins = _windows(4)
    allk = np.unique(np.concatenate(wins))
    C = 1 << 20
    assert len({store.entry_of(int(k), C) for k in allk}) == len(allk)  # no two share
    res = store.run_windows(wins, C, _fake_compute)
    seen = set()
    for w, r in enumerate(res):
        hits = {int(k) for k, p in zip(r["unique_keys"], r["miss_pos"]) if p < 0}
        assert hits == {int(k) for k in r["unique_keys"]} & seen, w
        seen |= {int(k) for k in r["unique_keys"]}
        assert r["n_miss"] == int((r["miss_pos"] >= 0).sum())
    assert res[0]["n_miss"] == len(res[0]["unique_keys"])
    assert res[1]["n_miss"] < len(res[1]["unique_keys"])   # hot templates recur


def test_one_entry_store_keeps_the_largest_missed_key():
    wins = [np.array([5, 9, 2, 9]), np.array([9, 1]), np.array([1, 3]), np.array([3, 20])]
    res = store.run_windows(wins, 1, _fake_compute)
    # window 0: all miss, 9 stored; window 1: 9 hits, 1 misses and replaces it
    assert list(res[0]["miss_pos"]) == [0, 1, 2]
    assert list(res[1]["miss_pos"]) == [0, -1]
    assert list(res[2]["miss_pos"]) == [-1, 0]      # 1 hit, 3 missed -> stored
    assert list(res[3]["miss_pos"]) == [-1, 0]      # 3 hit, 20 missed


def test_shared_entries_largest_key_wins():
    C = 8
    keys = list(range(1, 200))
    by_entry = {}
    for k in keys:
        by_entry.setdefault(store.entry_of(k, C), []).append(k)
    res = store.run_windows([np.array(keys), np.array(keys)], C, _fake_compute)
    hits = sorted(int(k) for k, p in zip(res[1]["unique_keys"], res[1]["miss_pos"]) if p < 0)
    assert hits == sorted(max(v) for v in by_entry.values())


def test_reused_rows_equal_fresh_results():
    # the distinct keys' rows of every window equal what the oracle computes
    # for them without any store (small corpus, real retrieval)
    wins = synth.window_stream("ridge1m", 3)
    c, _ = synth.gaussian_rows(wins[0].seed, synth.S_CORPUS, 700, 768, "bf16")
    k = 5

    def compute(w, miss_keys):
        ref = oracle.dedup(wins[w].keys)
        pos = np.searchsorted(ref["unique_keys"], miss_keys)
        rows = ref["first_index"][pos].astype(np.int64)
        return oracle.topk_exact(wins[w].q_req, c, k, q_rows=rows)

    for C in (1, 64, 4096):
        res = store.run_windows([w.keys for w in wins], C, compute)
        for w, r in enumerate(res):
            ref = oracle.dedup(wins[w].keys)
            np.testing.assert_array_equal(r["unique_keys"], ref["unique_keys"])
            fs, fi = oracle.topk_exact(wins[w].q_req, c, k,
                                       q_rows=ref["first_index"].astype(np.int64))
            np.testing.assert_array_equal(np.array(r["indices"]), fi)
            np.testing.assert_array_equal(np.array(r["scores"]), fs)
