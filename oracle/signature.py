"""ORACLE -- test infrastructure, not part of the product.

Node semantic signatures (HeraSys Eq. 2), hashed with SHA-256 as in the
paper's prototype (Sec. 4.1).  Eq. 2 names the ingredients -- operator type,
result-affecting parameters, input data, ordered predecessor signatures --
but not how they are combined into one hash input.  The reading taken here
(the same one the device implements, written independently below):

* message = le32(tau) | le32(len Theta) | Theta | le32(len D) | D |
  le32(m) | Sig(u_1) | ... | Sig(u_m), integers little-endian, so that no two
  different field tuples give the same message;
* D = the node's text, normalised for query-like nodes: ASCII letters folded
  to lower case, runs of ASCII whitespace collapsed to one space, leading and
  trailing whitespace dropped (bytes.lower / bytes.split / join);
* key = the digest's first 8 bytes, big-endian, as a signed int64.

SHA-256 itself is hashlib's (a library primitive).
"""
from __future__ import annotations

import hashlib
import struct
from typing import List, Optional, Sequence, Tuple

import numpy as np


def normalize(text: bytes) -> bytes:
    return b" ".join(bytes(text).lower().split())


def message(op_type: int, params: bytes, text: bytes, pred_digests: Sequence[bytes],
            normalize_text: bool) -> bytes:
    d = normalize(text) if normalize_text else bytes(text)
    p = bytes(params)
    return (struct.pack("<I", op_type) + struct.pack("<I", len(p)) + p +
            struct.pack("<I", len(d)) + d + struct.pack("<I", len(pred_digests)) +
            b"".join(bytes(x) for x in pred_digests))


def digest(op_type: int, params: bytes, text: bytes, pred_digests: Sequence[bytes] = (),
           normalize_text: bool = True) -> bytes:
    return hashlib.sha256(message(op_type, params, text, pred_digests, normalize_text)).digest()


def key_of(dig: bytes) -> int:
    return int.from_bytes(bytes(dig[:8]), "big", signed=True)


def signatures(op_type: np.ndarray, params: bytes, param_off: Optional[np.ndarray], text: bytes,
               text_off: Optional[np.ndarray], pred_off: Optional[np.ndarray],
               pred_idx: Optional[np.ndarray], levels: List[Tuple[int, int]],
               normalize_text: bool) -> Tuple[np.ndarray, np.ndarray]:
    """Digests [n, 32] uint8 and keys [n] int64 of nodes hashed level by level:
    `levels` lists (first, count) ranges in call order; a predecessor id
    outside [0, first) of its node's level stands for 32 zero bytes.  Rows of
    nodes in no level stay zero.  Offsets follow the device's clamping rule
    (a range is cut at its buffer's end; a reversed range is empty)."""
    n = len(op_type)
    dig = np.zeros((n, 32), dtype=np.uint8)
    keys = np.zeros(n, dtype=np.int64)

    def rng(off, i, size):
        if off is None:
            return 0, 0
        lo = min(max(int(off[i]), 0), size)
        hi = min(max(int(off[i + 1]), lo), size)
        return lo, hi

    n_pred = 0 if pred_idx is None else len(pred_idx)
    for first, count in levels:
        for v in range(first, first + count):
            a, b = rng(param_off, v, len(params))
            c, d = rng(text_off, v, len(text))
            preds = []
            if pred_off is not None:
                q0 = min(max(int(pred_off[v]), 0), n_pred)
                q1 = min(max(int(pred_off[v + 1]), q0), n_pred)
                for j in range(q0, q1):
                    u = int(pred_idx[j])
                    preds.append(dig[u].tobytes() if 0 <= u < first else bytes(32))
            h = digest(int(op_type[v]), params[a:b], text[c:d], preds, normalize_text)
            dig[v] = np.frombuffer(h, dtype=np.uint8)
            keys[v] = key_of(h)
    return dig, keys
