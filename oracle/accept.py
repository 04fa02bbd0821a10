"""ORACLE -- test infrastructure, not part of the product.

Acceptance rule for a floating-point top-k list against the exact oracle.

Scores are computed by the device with fp32 accumulation, so they may differ
from the exact values by rounding; the rule bounds that difference and only
asks for exact indices where the exact scores are separated by more than the
tolerance.  With tol(x) = 1e-3*|x| + 1e-6 (relative 1e-3 as specified for
fp32 accumulation, plus a small absolute floor so the bound is meaningful
near zero) and the oracle's order r_1..r_{k+1} with exact scores s(.):

  T1  |got_score_j - s(got_index_j)| <= tol(s(got_index_j))
  T2  got scores non-increasing; bit-equal neighbours in ascending index
  T3  indices distinct and in [0, N); slots beyond N hold (-inf, -1)
  T4  if s(r_k) - s(r_{k+1}) > tol(s(r_k)) the index sets are equal, and every
      rank j isolated by more than tol on both sides has got_index_j == r_j
  T5  every s(got_index_j) >= s(r_k) - tol(s(r_k))
"""
from __future__ import annotations

import numpy as np

REL = 1e-3
ABS = 1e-6


def tol(x):
    return REL * np.abs(x) + ABS


def check_topk(got_score, got_index, ref_score, ref_index, exact_of_got, N, k):
    """One query.  ref_* hold the oracle's k+1 best (exact fp64 scores);
    exact_of_got[j] is the oracle's exact score of got_index[j] (ignored for
    padding slots).  Returns a list of violation strings (empty = pass)."""
    bad = []
    got_score = np.asarray(got_score, dtype=np.float32)
    got_index = np.asarray(got_index, dtype=np.int64)
    nv = min(k, N)
    # T3
    if k > N:
        tail_s, tail_i = got_score[nv:], got_index[nv:]
        if not (np.all(np.isneginf(tail_s)) and np.all(tail_i == -1)):
            bad.append(f"T3 padding beyond N={N} not (-inf,-1): {tail_s}, {tail_i}")
    gi = got_index[:nv]
    gs = got_score[:nv]
    if np.any(gi < 0) or np.any(gi >= N):
        bad.append(f"T3 index out of range: {gi}")
        return bad
    if len(set(gi.tolist())) != nv:
        bad.append(f"T3 duplicate indices: {gi}")
    ex = np.asarray(exact_of_got, dtype=np.float64)[:nv]
    # T1
    err = np.abs(gs.astype(np.float64) - ex)
    over = err > tol(ex)
    if np.any(over):
        j = int(np.argmax(over))
        bad.append(f"T1 score error at rank {j}: got {gs[j]!r} exact {ex[j]!r}")
    # T2
    for j in range(nv - 1):
        if gs[j] < gs[j + 1]:
            bad.append(f"T2 not descending at {j}: {gs[j]} < {gs[j + 1]}")
            break
        if gs[j] == gs[j + 1] and gi[j] > gi[j + 1]:
            bad.append(f"T2 equal scores not in index order at {j}: {gi[j]} > {gi[j + 1]}")
            break
    rs = np.asarray(ref_score, dtype=np.float64)
    ri = np.asarray(ref_index, dtype=np.int64)
    if nv == 0:
        return bad
    sk = rs[nv - 1]
    # T5
    if np.any(ex < sk - tol(sk)):
        j = int(np.argmax(ex < sk - tol(sk)))
        bad.append(f"T5 rank {j} index {gi[j]} exact {ex[j]} below s(r_k)={sk}")
    # T4
    has_next = nv < N and ri.shape[0] > nv
    sk1 = rs[nv] if has_next else -np.inf
    if (not has_next) or (sk - sk1 > tol(sk)):
        if set(gi.tolist()) != set(ri[:nv].tolist()):
            bad.append(f"T4 set mismatch: got {sorted(gi.tolist())} want {sorted(ri[:nv].tolist())}")
    for j in range(nv):
        left = j == 0 or rs[j - 1] - rs[j] > tol(rs[j])
        nxt = rs[j + 1] if (j + 1 < rs.shape[0] and j + 1 < N) else -np.inf
        right = rs[j] - nxt > tol(rs[j])
        if left and right and gi[j] != ri[j]:
            bad.append(f"T4 isolated rank {j}: got {gi[j]} want {ri[j]}")
            break
    return bad


def check_all(got_score, got_index, ref_score, ref_index, exact_of_got, N, k, labels=None):
    """Apply check_topk row by row; returns list of (label, violations)."""
    out = []
    for t in range(got_score.shape[0]):
        v = check_topk(got_score[t], got_index[t], ref_score[t], ref_index[t],
                       exact_of_got[t], N, k)
        if v:
            out.append((labels[t] if labels is not None else t, v))
    return out
