"""ORACLE -- test infrastructure, not part of the product.

Reuse-driven priorities (HeraSys Eq. 3 and Eq. 7; Algorithm 1, phase 2),
written out in plain Python floats (IEEE binary64) and integers:

* phi*_g = sum of phi_v over the logical nodes merged into fused node g
  (Eq. 3).  Reading taken (the paper gives no precision): each phi_v, an fp32
  value clamped to [0, 2^16) with NaN as 0, is truncated to a multiple of
  2^-24 and the multiples are added exactly (Python integers), then the sum is
  rounded once to binary64;
* pi_g = alpha / (S + eps) + gamma * phi*_g + delta * y (Eq. 7), evaluated left
  to right in binary64, with S and y of the surviving node (the group's first
  request, to which the merged nodes are redirected, Sec. 3.3 (I));
* the ready-queue order: pi descending (the queues are keyed by pi,
  descending), equal pi by ascending group.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

UNIT = 1 << 24
PHI_MAX = np.float32(65535.99609375)      # largest fp32 below 2^16


def phi_units(phi: np.ndarray) -> list:
    """Per-request contributions in units of 2^-24 (clamped, NaN -> 0)."""
    out = []
    for f in np.asarray(phi, dtype=np.float32):
        v = float(f)
        if not v > 0.0:          # negative, zero or NaN
            out.append(0)
            continue
        v = min(v, float(PHI_MAX))
        out.append(math.floor(v * UNIT))   # v * 2^24 is exact in binary64
    return out


def priorities(inverse: np.ndarray, first_index: np.ndarray, phi: np.ndarray,
               s_hat: np.ndarray, heavy: Optional[np.ndarray], alpha: float, gamma: float,
               delta: float, eps: float):
    """(phi_fused [n_u] float64, pi [n_u] float64, order [n_u] int32)."""
    n_u = len(first_index)
    units = [0] * n_u
    for i, u in enumerate(phi_units(phi)):
        units[int(inverse[i])] += u
    phi_f = np.array([float(u) / UNIT for u in units], dtype=np.float64)
    pi = np.empty(n_u, dtype=np.float64)
    for g in range(n_u):
        s = int(first_index[g])
        sq = float(np.float32(s_hat[s]))
        y = 1.0 if (heavy is not None and heavy[s]) else 0.0
        p = alpha / (sq + eps) + gamma * float(phi_f[g]) + delta * y
        pi[g] = 0.0 if p == 0.0 else p
    order = sorted(range(n_u), key=lambda g: (-pi[g], g))
    return phi_f, pi, np.array(order, dtype=np.int32)
