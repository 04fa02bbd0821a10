"""ORACLE -- test infrastructure, not part of the product.

Python wrapper around liboracle.so (oracle.c): the plain CPU reference for
merged retrieval (dedup by signature, exact fp64 inner-product top-k with ties
to the lower chunk index, delivery of each distinct result to every request
carrying the same signature).  Only tests/, the smoke check and the
benchmark's CPU-baseline leg import this package.  It never imports the GPU
package and shares no code with it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None

ENC = {"f32": 0, "bf16": 1, "fp8": 2}


def build(verbose: bool = False) -> str:
    src = os.path.join(_HERE, "oracle.c")
    tmp = _SO + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", src, "-lm", "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_SO):
        build()
    lib = ctypes.CDLL(_SO)
    i64, i32, vp, dbl = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_double
    lib.or_e4m3_decode.argtypes = [ctypes.c_uint8]
    lib.or_e4m3_decode.restype = dbl
    lib.or_bf16_decode.argtypes = [ctypes.c_uint16]
    lib.or_bf16_decode.restype = dbl
    lib.or_dedup.argtypes = [vp, i64, vp, vp, vp, vp, vp]
    lib.or_dedup.restype = i32
    lib.or_gather_rows.argtypes = [vp, i64, i64, vp, i32, i64, vp]
    lib.or_gather_rows.restype = i32
    lib.or_topk_exact.argtypes = [vp, i32, i64, vp, vp, i32, vp, i64, i64, i64, vp, vp, i32]
    lib.or_topk_exact.restype = i32
    lib.or_score_pairs.argtypes = [vp, i32, vp, i32, vp, i64, i64, vp, vp, vp, i32]
    lib.or_score_pairs.restype = i32
    lib.or_merge_retrieval.argtypes = ([vp, i64, vp, i32, vp, i32, vp, i64, i64, i64, i64, vp]
                                       + [vp] * 9 + [i32])
    lib.or_merge_retrieval.restype = i32
    _lib = lib
    return lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def enc_of(a: np.ndarray) -> str:
    """Storage encoding of an array: float32 -> f32, uint16 -> bf16 bits,
    uint8 -> e4m3 codes."""
    return {np.dtype(np.float32): "f32", np.dtype(np.uint16): "bf16",
            np.dtype(np.uint8): "fp8"}[a.dtype]


def e4m3_decode(code: int) -> float:
    return _load().or_e4m3_decode(code)


def bf16_decode(bits: int) -> float:
    return _load().or_bf16_decode(bits)


def dedup(keys: np.ndarray) -> dict:
    keys = np.ascontiguousarray(keys, dtype=np.int64)
    R = keys.shape[0]
    uk = np.zeros(max(R, 1), np.int64)
    fi = np.zeros(max(R, 1), np.int32)
    ct = np.zeros(max(R, 1), np.int32)
    inv = np.zeros(max(R, 1), np.int32)
    nu = np.zeros(1, np.int64)
    if _load().or_dedup(_p(keys), R, _p(uk), _p(fi), _p(ct), _p(inv), _p(nu)) != 0:
        raise RuntimeError("or_dedup failed")
    n = int(nu[0])
    return {"n_unique": n, "unique_keys": uk[:n], "first_index": fi[:n],
            "counts": ct[:n], "inverse": inv[:R]}


def gather_rows(src: np.ndarray, index: np.ndarray) -> np.ndarray:
    src = np.ascontiguousarray(src)
    index = np.ascontiguousarray(index)
    is64 = 1 if index.dtype == np.int64 else 0
    if not is64:
        index = index.astype(np.int32)
    rows = src.shape[0]
    row_bytes = src.nbytes // max(rows, 1) if rows else 0
    out = np.empty((index.shape[0],) + src.shape[1:], dtype=src.dtype)
    if _load().or_gather_rows(_p(src), rows, row_bytes, _p(index), is64, index.shape[0],
                              _p(out)) != 0:
        raise IndexError("or_gather_rows: index out of range")
    return out


def topk_exact(Q: np.ndarray, C: np.ndarray, kk: int, scale: Optional[np.ndarray] = None,
               q_rows: Optional[np.ndarray] = None, threads: Optional[int] = None):
    """Exact top-kk (score desc, index asc) of each selected query row.
    Returns (scores float64 [n, kk], index int64 [n, kk])."""
    Q = np.ascontiguousarray(Q)
    C = np.ascontiguousarray(C)
    d = Q.shape[1]
    assert C.shape[1] == d
    ce = enc_of(C)
    if ce == "fp8":
        assert scale is not None
        scale = np.ascontiguousarray(scale, dtype=np.float32)
    if q_rows is not None:
        q_rows = np.ascontiguousarray(q_rows, dtype=np.int64)
        n = q_rows.shape[0]
    else:
        n = Q.shape[0]
    bs = np.empty((n, kk), np.float64)
    bi = np.empty((n, kk), np.int64)
    rc = _load().or_topk_exact(_p(Q), ENC[enc_of(Q)], n, _p(q_rows), _p(C), ENC[ce], _p(scale),
                               C.shape[0], d, kk, _p(bs), _p(bi), threads or default_threads())
    if rc != 0:
        raise RuntimeError("or_topk_exact failed")
    return bs, bi


def score_pairs(Q: np.ndarray, C: np.ndarray, q_idx: np.ndarray, c_idx: np.ndarray,
                scale: Optional[np.ndarray] = None, threads: Optional[int] = None) -> np.ndarray:
    Q = np.ascontiguousarray(Q)
    C = np.ascontiguousarray(C)
    q_idx = np.ascontiguousarray(q_idx, dtype=np.int64).ravel()
    c_idx = np.ascontiguousarray(c_idx, dtype=np.int64).ravel()
    assert q_idx.shape == c_idx.shape
    if scale is not None:
        scale = np.ascontiguousarray(scale, dtype=np.float32)
    out = np.empty(q_idx.shape[0], np.float64)
    rc = _load().or_score_pairs(_p(Q), ENC[enc_of(Q)], _p(C), ENC[enc_of(C)], _p(scale),
                                Q.shape[1], q_idx.shape[0], _p(q_idx), _p(c_idx), _p(out),
                                threads or default_threads())
    if rc != 0:
        raise RuntimeError("or_score_pairs failed")
    return out


def merge_retrieval(keys: np.ndarray, q_req: np.ndarray, corpus: np.ndarray, k: int,
                    scale: Optional[np.ndarray] = None, u_sel: Optional[np.ndarray] = None,
                    threads: Optional[int] = None) -> dict:
    """The whole path: dedup, representative rows, exact top-k of the distinct
    rows (all, or the distinct positions listed in u_sel), delivery to every
    request.  Requests whose group is not selected get out rows of (nan, -2)."""
    keys = np.ascontiguousarray(keys, dtype=np.int64)
    q_req = np.ascontiguousarray(q_req)
    corpus = np.ascontiguousarray(corpus)
    R, d = q_req.shape
    N = corpus.shape[0]
    if scale is not None:
        scale = np.ascontiguousarray(scale, dtype=np.float32)
    if u_sel is not None:
        u_sel = np.ascontiguousarray(u_sel, dtype=np.int64)
    n_sel = 0 if u_sel is None else u_sel.shape[0]
    cap = max(R, 1)
    uk = np.zeros(cap, np.int64)
    fi = np.zeros(cap, np.int32)
    ct = np.zeros(cap, np.int32)
    inv = np.zeros(cap, np.int32)
    nu = np.zeros(1, np.int64)
    nsel_cap = max(cap if u_sel is None else n_sel, 1)
    us = np.zeros((nsel_cap, k), np.float32)
    ui = np.zeros((nsel_cap, k), np.int32)
    os_ = np.full((cap, k), np.nan, np.float32)
    oi = np.full((cap, k), -2, np.int32)
    rc = _load().or_merge_retrieval(
        _p(keys), R, _p(q_req), ENC[enc_of(q_req)], _p(corpus), ENC[enc_of(corpus)], _p(scale),
        N, d, k, n_sel, _p(u_sel), _p(uk), _p(fi), _p(ct), _p(inv), _p(nu), _p(us), _p(ui),
        _p(os_), _p(oi), threads or default_threads())
    if rc != 0:
        raise RuntimeError("or_merge_retrieval failed")
    n = int(nu[0])
    ns = n if u_sel is None else n_sel
    return {"n_unique": n, "unique_keys": uk[:n], "first_index": fi[:n], "counts": ct[:n],
            "inverse": inv[:R], "u_score": us[:ns], "u_index": ui[:ns],
            "out_score": os_[:R], "out_index": oi[:R]}
