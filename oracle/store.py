"""ORACLE -- test infrastructure, not part of the product.

Model of cross-window result reuse (HeraSys Sec. 3.3 (II), asynchronous cache
reuse): a retrieval node whose signature equals that of a node completed in
an earlier window takes the stored result instead of being executed again.

The paper does not say how many results are kept or which one gives way when
the store is full.  The reading taken here (the same one the device store
implements, written independently below from its definition):

* the store has C = 2^b entries; key -> entry by Fibonacci hashing, i.e.
  Knuth's multiplicative hashing with the multiplier floor(2^64 / phi):
  entry = the top b bits of (key * multiplier) mod 2^64 (key taken as its
  64-bit two's-complement pattern);
* a key hits when its entry holds a result for that same key;
* after a window, every missed key is written to its entry; where several
  missed keys of the window share an entry, the largest key wins; a write
  replaces what the entry held.

Plain Python over dicts: slow and obviously correct, meant for a few thousand
keys per window.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Tuple

import numpy as np

# floor(2^64 / golden ratio), the multiplier of Fibonacci hashing
FIB_MULT = 11400714819323198485


def entry_of(key: int, capacity: int) -> int:
    """Entry of `key` in a store of `capacity` = 2^b entries."""
    if capacity < 1 or capacity & (capacity - 1):
        raise ValueError("capacity must be a power of two")
    b = capacity.bit_length() - 1
    if b == 0:
        return 0
    h = ((int(key) % (1 << 64)) * FIB_MULT) % (1 << 64)
    return h >> (64 - b)


class StoreModel:
    """Entries: entry -> (key, score row, index row)."""

    def __init__(self, capacity: int):
        entry_of(0, capacity)   # validates
        self.capacity = capacity
        self.entries: Dict[int, Tuple[int, np.ndarray, np.ndarray]] = {}

    def lookup(self, unique_keys) -> Tuple[np.ndarray, int]:
        """miss_pos[u] = -1 for a hit, else the miss's rank among the
        window's misses in the order of `unique_keys`; returns (miss_pos,
        number of misses)."""
        miss_pos = np.full(len(unique_keys), -1, dtype=np.int64)
        n = 0
        for u, key in enumerate(unique_keys):
            e = self.entries.get(entry_of(int(key), self.capacity))
            if e is None or e[0] != int(key):
                miss_pos[u] = n
                n += 1
        return miss_pos, n

    def stored(self, key: int):
        e = self.entries.get(entry_of(int(key), self.capacity))
        if e is None or e[0] != int(key):
            return None
        return e[1], e[2]

    def insert(self, unique_keys, miss_pos, scores, indices):
        """Writes the window's missed keys (rows of scores/indices by
        position in `unique_keys`)."""
        winner: Dict[int, int] = {}
        for u, key in enumerate(unique_keys):
            if miss_pos[u] < 0:
                continue
            e = entry_of(int(key), self.capacity)
            if e not in winner or int(key) > int(unique_keys[winner[e]]):
                winner[e] = u
        for e, u in winner.items():
            self.entries[e] = (int(unique_keys[u]), np.array(scores[u]), np.array(indices[u]))


def run_windows(windows: List[np.ndarray], capacity: int,
                compute: Callable[[int, np.ndarray], Tuple[np.ndarray, np.ndarray]]):
    """Distinct keys of every window (ascending), looked up in the store,
    misses computed by compute(window, miss_keys) -> (scores, indices) and
    inserted.  Returns per window a dict with unique_keys, miss_pos, n_miss,
    and the window's full (scores, indices) rows."""
    store = StoreModel(capacity)
    out = []
    for w, keys in enumerate(windows):
        uk = np.unique(np.asarray(keys, dtype=np.int64))
        miss_pos, n_miss = store.lookup(uk)
        miss_keys = uk[miss_pos >= 0]
        ms, mi = compute(w, miss_keys)
        rows_s, rows_i = [None] * len(uk), [None] * len(uk)
        for u, key in enumerate(uk):
            if miss_pos[u] >= 0:
                rows_s[u], rows_i[u] = ms[miss_pos[u]], mi[miss_pos[u]]
            else:
                rows_s[u], rows_i[u] = store.stored(int(key))
        store.insert(uk, miss_pos, rows_s, rows_i)
        out.append(dict(unique_keys=uk, miss_pos=miss_pos, n_miss=n_miss,
                        scores=rows_s, indices=rows_i))
    return out
