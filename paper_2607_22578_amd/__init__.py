"""Python binding of libhsmerge.so (merged retrieval on MI355X / gfx950).

Argument marshalling only: every step runs in the HIP kernels of the shared
library.  Functions carry the C names of include/hs_merge.h and take device
buffers as torch tensors (or raw integer addresses); PyTorch serves only to
own device memory and streams.  Importing fails loudly when the library has
not been built -- there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhsmerge.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(hipcc --offload-arch=gfx950)")

# torch ships its own HIP runtime.  Load it first so that the library binds to
# the same runtime instance (by soname) instead of bringing a second runtime
# into the process; two runtimes cannot share the device.
try:
    import torch as _torch  # noqa: F401
except ImportError:  # plain C-ABI use without torch
    _torch = None

_lib = ctypes.CDLL(LIB_PATH)

HS_OK, HS_ERR_INVALID_ARG, HS_ERR_UNSUPPORTED, HS_ERR_WORKSPACE, HS_ERR_ALIGNMENT, \
    HS_ERR_DEVICE = range(6)
HS_F32, HS_BF16, HS_FP8_E4M3 = 0, 1, 2
ABI_VERSION = 3

EXPORTS = ["hs_merge_plan", "hs_plan_destroy", "hs_workflow_rows", "hs_dedup", "hs_score_topk",
           "hs_score_topk_noalloc", "hs_score_partial", "hs_topk_merge", "hs_corpus_tiled_bytes",
           "hs_tile_corpus", "hs_scatter", "hs_deliver",
           "hs_cache_bytes", "hs_cache_reset", "hs_cache_lookup",
           "hs_cache_insert", "hs_signature", "hs_priority", "hs_status_string",
           "hs_last_error", "hs_abi_version"]
HS_SIG_NORMALIZE_TEXT = 1
HS_FLAG_TILED_CORPUS = 1


class hs_merge_desc(ctypes.Structure):
    _fields_ = [("n_requests", ctypes.c_int64), ("dim", ctypes.c_int64),
                ("n_corpus", ctypes.c_int64), ("k", ctypes.c_int32),
                ("query_dtype", ctypes.c_int32), ("corpus_dtype", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("max_unique", ctypes.c_int64),
                ("n_workflows", ctypes.c_int64),
                ("workflow_offsets", ctypes.POINTER(ctypes.c_int64))]


class hs_sig_nodes(ctypes.Structure):
    _fields_ = [("op_type", ctypes.c_void_p), ("params", ctypes.c_void_p),
                ("param_off", ctypes.c_void_p), ("param_bytes", ctypes.c_int64),
                ("text", ctypes.c_void_p), ("text_off", ctypes.c_void_p),
                ("text_bytes", ctypes.c_int64), ("pred_off", ctypes.c_void_p),
                ("pred_idx", ctypes.c_void_p), ("pred_count", ctypes.c_int64),
                ("n_nodes", ctypes.c_int64)]


_vp, _i64, _i32, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
_lib.hs_merge_plan.argtypes = [ctypes.POINTER(hs_merge_desc), ctypes.POINTER(_vp),
                               ctypes.POINTER(_sz)]
_lib.hs_merge_plan.restype = ctypes.c_int
_lib.hs_plan_destroy.argtypes = [_vp]
_lib.hs_plan_destroy.restype = None
_lib.hs_workflow_rows.argtypes = [_vp, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i64)]
_lib.hs_workflow_rows.restype = ctypes.c_int
_lib.hs_deliver.argtypes = [_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp]
_lib.hs_deliver.restype = ctypes.c_int
_lib.hs_dedup.argtypes = [_vp] + [_vp] * 7 + [_vp, _sz, _vp]
_lib.hs_dedup.restype = ctypes.c_int
_lib.hs_score_topk.argtypes = [_vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.hs_score_topk.restype = ctypes.c_int
_lib.hs_score_topk_noalloc.argtypes = [_vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp]
_lib.hs_score_topk_noalloc.restype = ctypes.c_int
_lib.hs_score_partial.argtypes = [_vp, _vp, _i64, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.hs_score_partial.restype = ctypes.c_int
_lib.hs_topk_merge.argtypes = [_vp, _i64, _vp, _vp, _vp, _vp, _sz, _vp]
_lib.hs_topk_merge.restype = ctypes.c_int
_lib.hs_corpus_tiled_bytes.argtypes = [_vp, ctypes.POINTER(_sz)]
_lib.hs_corpus_tiled_bytes.restype = ctypes.c_int
_lib.hs_tile_corpus.argtypes = [_vp, _vp, _vp, _sz, _vp]
_lib.hs_tile_corpus.restype = ctypes.c_int
_lib.hs_scatter.argtypes = [_vp, _i64, _i64, _vp, _i32, _i64, _vp, _vp, _vp]
_lib.hs_scatter.restype = ctypes.c_int
_lib.hs_cache_bytes.argtypes = [_vp, _i64, ctypes.POINTER(_sz)]
_lib.hs_cache_bytes.restype = ctypes.c_int
_lib.hs_cache_reset.argtypes = [_vp, _vp, _sz, _i64, _vp]
_lib.hs_cache_reset.restype = ctypes.c_int
_lib.hs_cache_lookup.argtypes = [_vp, _vp, _sz, _i64, _vp, _vp, _i64] + [_vp] * 7
_lib.hs_cache_lookup.restype = ctypes.c_int
_lib.hs_cache_insert.argtypes = [_vp, _vp, _sz, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp]
_lib.hs_cache_insert.restype = ctypes.c_int
_lib.hs_signature.argtypes = [ctypes.POINTER(hs_sig_nodes), _i64, _i64, _i32, _vp, _vp, _vp]
_lib.hs_signature.restype = ctypes.c_int
_dbl = ctypes.c_double
_lib.hs_priority.argtypes = ([_vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _dbl, _dbl, _dbl, _dbl]
                             + [_vp] * 4 + [_sz, _vp])
_lib.hs_priority.restype = ctypes.c_int
_lib.hs_status_string.argtypes = [ctypes.c_int]
_lib.hs_status_string.restype = ctypes.c_char_p
_lib.hs_last_error.argtypes = []
_lib.hs_last_error.restype = ctypes.c_char_p
_lib.hs_abi_version.argtypes = []
_lib.hs_abi_version.restype = ctypes.c_int32


class HsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{hs_status_string(status)}: {msg}")
        self.status = status


def hs_status_string(status: int) -> str:
    return _lib.hs_status_string(status).decode()


def hs_last_error() -> str:
    return _lib.hs_last_error().decode()


def hs_abi_version() -> int:
    return int(_lib.hs_abi_version())


def _check(status: int):
    if status != HS_OK:
        raise HsError(status, hs_last_error())


def _ptr(x):
    """Device/host address of a torch tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def dtype_code(t) -> int:
    """HS dtype of a torch tensor (float32, bfloat16, uint8/float8_e4m3fn)."""
    import torch
    m = {torch.float32: HS_F32, torch.bfloat16: HS_BF16, torch.uint8: HS_FP8_E4M3,
         torch.float8_e4m3fn: HS_FP8_E4M3}
    if t.dtype not in m:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return m[t.dtype]


@dataclass
class Plan:
    handle: int
    workspace_bytes: int
    desc: hs_merge_desc

    def __del__(self):
        # (at interpreter exit the module's globals may already be gone)
        if self.handle and _lib is not None:
            _lib.hs_plan_destroy(self.handle)
            self.handle = 0


def hs_merge_plan(n_requests: int, dim: int, n_corpus: int, k: int, query_dtype: int,
                  corpus_dtype: int, max_unique: int = 0, flags: int = 0,
                  n_workflows: int = 1, workflow_offsets=None) -> Plan:
    """workflow_offsets: None (uniform) or a sequence of n_workflows + 1
    request offsets (host CSR)."""
    off = None
    if workflow_offsets is not None:
        vals = [int(x) for x in workflow_offsets]
        off = (ctypes.c_int64 * max(len(vals), 1))(*vals)
    d = hs_merge_desc(n_requests, dim, n_corpus, k, query_dtype, corpus_dtype, flags, max_unique,
                      n_workflows, ctypes.cast(off, ctypes.POINTER(ctypes.c_int64))
                      if off is not None else None)
    h = _vp()
    ws = _sz()
    _check(_lib.hs_merge_plan(ctypes.byref(d), ctypes.byref(h), ctypes.byref(ws)))
    d.workflow_offsets = None   # the plan keeps its own copy
    return Plan(h.value, int(ws.value), d)


def hs_workflow_rows(plan: Plan, w: int):
    """(first, count): rows of workflow w in the per-request outputs."""
    a, b = _i64(), _i64()
    _check(_lib.hs_workflow_rows(plan.handle, w, ctypes.byref(a), ctypes.byref(b)))
    return int(a.value), int(b.value)


def hs_deliver(plan: Plan, topk_score, topk_index, topk_rows: int, inverse, out_score, out_index,
               stream=None):
    _check(_lib.hs_deliver(plan.handle, _ptr(topk_score), _ptr(topk_index), topk_rows,
                           _ptr(inverse), _ptr(out_score), _ptr(out_index), _stream(stream)))


def hs_dedup(plan: Plan, keys, unique_keys, first_index, counts, inverse, n_unique_dev,
             n_unique_host=None, ws=None, ws_bytes: Optional[int] = None, stream=None):
    host = None
    if n_unique_host is True:
        host = ctypes.c_int64(-1)
        hptr = ctypes.addressof(host)
    else:
        hptr = _ptr(n_unique_host)
    _check(_lib.hs_dedup(plan.handle, _ptr(keys), _ptr(unique_keys), _ptr(first_index),
                         _ptr(counts), _ptr(inverse), _ptr(n_unique_dev), hptr, _ptr(ws),
                         _ws_bytes(ws, ws_bytes), _stream(stream)))
    return None if host is None else int(host.value)


def _ws_bytes(ws, ws_bytes):
    if ws_bytes is not None:
        return ws_bytes
    if ws is None or isinstance(ws, int):
        return 0
    return ws.numel() * ws.element_size()


def hs_score_topk(plan: Plan, q_unique, n_unique: int, n_unique_dev, corpus, row_scale,
                  topk_score, topk_index, ws=None, ws_bytes: Optional[int] = None, stream=None):
    _check(_lib.hs_score_topk(plan.handle, _ptr(q_unique), n_unique, _ptr(n_unique_dev),
                              _ptr(corpus), _ptr(row_scale), _ptr(topk_score), _ptr(topk_index),
                              _ptr(ws), _ws_bytes(ws, ws_bytes), _stream(stream)))


def hs_corpus_tiled_bytes(plan: Plan) -> int:
    n = _sz()
    _check(_lib.hs_corpus_tiled_bytes(plan.handle, ctypes.byref(n)))
    return int(n.value)


def hs_tile_corpus(plan: Plan, corpus, tiled, tiled_bytes: Optional[int] = None, stream=None):
    if tiled_bytes is None:
        tiled_bytes = tiled.numel() * tiled.element_size() if tiled is not None else 0
    _check(_lib.hs_tile_corpus(plan.handle, _ptr(corpus), _ptr(tiled), tiled_bytes,
                               _stream(stream)))


def hs_score_topk_noalloc(plan: Plan, q_unique, n_unique: int, n_unique_dev, corpus, row_scale,
                          topk_score, topk_index, stream=None):
    _check(_lib.hs_score_topk_noalloc(plan.handle, _ptr(q_unique), n_unique, _ptr(n_unique_dev),
                                      _ptr(corpus), _ptr(row_scale), _ptr(topk_score),
                                      _ptr(topk_index), _stream(stream)))


def hs_score_partial(plan: Plan, q_unique, n_unique: int, n_unique_dev, corpus, row_scale,
                     ws=None, ws_bytes: Optional[int] = None, stream=None):
    _check(_lib.hs_score_partial(plan.handle, _ptr(q_unique), n_unique, _ptr(n_unique_dev),
                                 _ptr(corpus), _ptr(row_scale), _ptr(ws),
                                 _ws_bytes(ws, ws_bytes), _stream(stream)))


def hs_topk_merge(plan: Plan, n_unique: int, n_unique_dev, topk_score, topk_index, ws=None,
                  ws_bytes: Optional[int] = None, stream=None):
    _check(_lib.hs_topk_merge(plan.handle, n_unique, _ptr(n_unique_dev), _ptr(topk_score),
                              _ptr(topk_index), _ptr(ws), _ws_bytes(ws, ws_bytes),
                              _stream(stream)))


def hs_scatter(src, src_rows: int, row_bytes: int, index, index_is_i64: int, n_out: int,
               n_out_dev, dst, stream=None):
    _check(_lib.hs_scatter(_ptr(src), src_rows, row_bytes, _ptr(index), index_is_i64, n_out,
                           _ptr(n_out_dev), _ptr(dst), _stream(stream)))


def hs_cache_bytes(plan: Plan, capacity: int) -> int:
    b = _sz()
    _check(_lib.hs_cache_bytes(plan.handle, capacity, ctypes.byref(b)))
    return int(b.value)


def hs_cache_reset(plan: Plan, cache, capacity: int, cache_bytes: Optional[int] = None,
                   stream=None):
    _check(_lib.hs_cache_reset(plan.handle, _ptr(cache), _ws_bytes(cache, cache_bytes), capacity,
                               _stream(stream)))


def hs_cache_lookup(plan: Plan, cache, capacity: int, unique_keys, first_index, n_unique: int,
                    n_unique_dev, topk_score, topk_index, miss_pos, miss_first, n_miss_dev,
                    cache_bytes: Optional[int] = None, stream=None):
    _check(_lib.hs_cache_lookup(plan.handle, _ptr(cache), _ws_bytes(cache, cache_bytes), capacity,
                                _ptr(unique_keys), _ptr(first_index), n_unique,
                                _ptr(n_unique_dev), _ptr(topk_score), _ptr(topk_index),
                                _ptr(miss_pos), _ptr(miss_first), _ptr(n_miss_dev),
                                _stream(stream)))


def hs_cache_insert(plan: Plan, cache, capacity: int, unique_keys, miss_pos, n_unique: int,
                    n_unique_dev, topk_score, topk_index, cache_bytes: Optional[int] = None,
                    stream=None):
    _check(_lib.hs_cache_insert(plan.handle, _ptr(cache), _ws_bytes(cache, cache_bytes), capacity,
                                _ptr(unique_keys), _ptr(miss_pos), n_unique, _ptr(n_unique_dev),
                                _ptr(topk_score), _ptr(topk_index), _stream(stream)))


def _nbytes(x):
    if x is None or isinstance(x, int):
        return 0
    return x.numel() * x.element_size()


def hs_signature(op_type, n_nodes: int, first: int, count: int, digest, keys=None, params=None,
                 param_off=None, text=None, text_off=None, pred_off=None, pred_idx=None,
                 flags: int = 0, param_bytes: Optional[int] = None,
                 text_bytes: Optional[int] = None, pred_count: Optional[int] = None,
                 stream=None):
    """Signatures of nodes [first, first + count) (digests and 64-bit keys);
    buffer sizes default to the tensors' sizes."""
    nd = hs_sig_nodes(_ptr(op_type), _ptr(params), _ptr(param_off),
                      _nbytes(params) if param_bytes is None else param_bytes,
                      _ptr(text), _ptr(text_off), _nbytes(text) if text_bytes is None else text_bytes,
                      _ptr(pred_off), _ptr(pred_idx),
                      (_nbytes(pred_idx) // 4) if pred_count is None else pred_count, n_nodes)
    _check(_lib.hs_signature(ctypes.byref(nd), first, count, flags, _ptr(digest), _ptr(keys),
                             _stream(stream)))


def hs_priority(plan: Plan, inverse, first_index, n_unique: int, n_unique_dev, phi, s_hat, heavy,
                alpha: float, gamma: float, delta: float, eps: float, phi_fused, pi, order,
                ws=None, ws_bytes: Optional[int] = None, stream=None):
    _check(_lib.hs_priority(plan.handle, _ptr(inverse), _ptr(first_index), n_unique,
                            _ptr(n_unique_dev), _ptr(phi), _ptr(s_hat), _ptr(heavy), alpha, gamma,
                            delta, eps, _ptr(phi_fused), _ptr(pi), _ptr(order), _ptr(ws),
                            _ws_bytes(ws, ws_bytes), _stream(stream)))


# ---------------------------------------------------------------- composition

class MergedRetrieval:
    """Owns the plan, workspace and per-window buffers for one shape and runs
    the whole path (dedup -> representative rows -> score/top-k -> delivery)
    on one stream.  All outputs are torch tensors on the device."""

    def __init__(self, n_requests: int, dim: int, n_corpus: int, k: int, query_dtype: int,
                 corpus_dtype: int, device="cuda", max_unique: int = 0, n_workflows: int = 1,
                 workflow_offsets=None, tiled_corpus: bool = False):
        """tiled_corpus: the score calls take the corpus in the tiled layout
        (make it once with tile_corpus)."""
        import torch
        self.R, self.d, self.N, self.k = n_requests, dim, n_corpus, k
        self.qdt, self.cdt = query_dtype, corpus_dtype
        self.tiled_corpus = tiled_corpus
        self.plan = hs_merge_plan(n_requests, dim, n_corpus, k, query_dtype, corpus_dtype,
                                  max_unique, flags=HS_FLAG_TILED_CORPUS if tiled_corpus else 0,
                                  n_workflows=n_workflows,
                                  workflow_offsets=workflow_offsets)
        self.n_workflows = n_workflows
        cap = max_unique if max_unique > 0 else n_requests
        self.cap = cap
        dev = torch.device(device)
        R1 = max(n_requests, 1)
        qt = torch.float32 if query_dtype == HS_F32 else torch.bfloat16
        self.ws = torch.empty(max(self.plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
        self.unique_keys = torch.empty(R1, dtype=torch.int64, device=dev)
        self.first_index = torch.empty(R1, dtype=torch.int32, device=dev)
        self.counts = torch.empty(R1, dtype=torch.int32, device=dev)
        self.inverse = torch.empty(R1, dtype=torch.int32, device=dev)
        self.n_unique = torch.zeros(1, dtype=torch.int64, device=dev)
        # rows for every distinct query of a window (more than one batch of
        # max_unique when the window has more distinct keys)
        self.q_unique = torch.empty((R1, dim), dtype=qt, device=dev)
        self.topk_score = torch.empty((R1, k), dtype=torch.float32, device=dev)
        self.topk_index = torch.empty((R1, k), dtype=torch.int32, device=dev)
        self.out_score = torch.empty((R1, k), dtype=torch.float32, device=dev)
        self.out_index = torch.empty((R1, k), dtype=torch.int32, device=dev)
        self.q_row_bytes = dim * (4 if query_dtype == HS_F32 else 2)

    def tile_corpus(self, corpus, stream=None):
        """The tiled copy of a row-major BF16/FP8 corpus (a new device tensor),
        for a MergedRetrieval made with tiled_corpus=True."""
        import torch
        out = torch.empty(max(hs_corpus_tiled_bytes(self.plan), 16), dtype=torch.uint8,
                          device=corpus.device)
        hs_tile_corpus(self.plan, corpus, out, stream=stream)
        return out

    def dedup(self, keys, stream=None, host_count: bool = False):
        return hs_dedup(self.plan, keys, self.unique_keys, self.first_index, self.counts,
                        self.inverse, self.n_unique, True if host_count else None, self.ws,
                        stream=stream)

    def gather_queries(self, q_req, stream=None):
        hs_scatter(q_req, self.R, self.q_row_bytes, self.first_index, 0, self.cap,
                   self.n_unique, self.q_unique, stream=stream)

    def score_partial(self, corpus, scale=None, n_unique: int = -1, stream=None):
        hs_score_partial(self.plan, self.q_unique, n_unique, self.n_unique, corpus, scale,
                         self.ws, stream=stream)

    def topk_merge(self, n_unique: int = -1, stream=None):
        hs_topk_merge(self.plan, n_unique, self.n_unique, self.topk_score, self.topk_index,
                      self.ws, stream=stream)

    def deliver(self, stream=None):
        hs_deliver(self.plan, self.topk_score, self.topk_index, self.topk_score.shape[0],
                   self.inverse, self.out_score, self.out_index, stream=stream)

    def workflow_results(self, w: int):
        """(scores, indices) of workflow w's requests: views of its rows of
        the per-request outputs."""
        first, count = hs_workflow_rows(self.plan, w)
        return (self.out_score[first:first + count], self.out_index[first:first + count])

    def run(self, keys, q_req, corpus, scale=None, stream=None, n_unique: int = -1):
        """The whole window; n_unique = -1 keeps the distinct count on the
        device (no host synchronisation).  With max_unique below the number
        of requests, the distinct count is read on the host (one
        synchronisation) and the distinct queries are scored in batches of at
        most max_unique (B_r), so that no group is left unscored."""
        if self.cap < self.R:
            nu = self.dedup(keys, stream, host_count=True)
            hs_scatter(q_req, self.R, self.q_row_bytes, self.first_index, 0, self.R,
                       self.n_unique, self.q_unique, stream=stream)
            self.score_chunked(corpus, nu, self.cap, scale, stream)
            self.deliver(stream)
            return
        self.dedup(keys, stream)
        self.gather_queries(q_req, stream)
        self.score_partial(corpus, scale, n_unique, stream)
        self.topk_merge(n_unique, stream)
        self.deliver(stream)

    # ------------------------------------------------ cross-window reuse

    def enable_cache(self, capacity: int, stream=None):
        """Allocates and empties a result store of `capacity` entries (a
        power of two) and the per-window miss buffers of run_cached."""
        import torch
        dev = self.ws.device
        self.cache_capacity = capacity
        self.cache = torch.empty(max(hs_cache_bytes(self.plan, capacity), 256), dtype=torch.uint8,
                                 device=dev)
        c1 = max(self.cap, 1)
        self.miss_pos = torch.empty(c1, dtype=torch.int32, device=dev)
        self.miss_first = torch.empty(c1, dtype=torch.int32, device=dev)
        self.n_miss = torch.zeros(1, dtype=torch.int64, device=dev)
        self.q_miss = torch.empty_like(self.q_unique)
        self.miss_score = torch.empty_like(self.topk_score)
        self.miss_index = torch.empty_like(self.topk_index)
        hs_cache_reset(self.plan, self.cache, capacity, stream=stream)

    def run_cached(self, keys, q_req, corpus, scale=None, stream=None, score_events=None):
        """The whole window with reuse of earlier windows' results: dedup ->
        store lookup (hit rows filled) -> representative rows of the misses ->
        score/top-k of the misses -> miss rows put in place -> store insert ->
        delivery.  Distinct and miss counts stay on the device.  score_events
        = (start, end) events recorded around the score step, if given."""
        if self.cap < self.R:
            raise ValueError("run_cached scores one batch per window: it needs max_unique = 0 "
                             "(or n_requests)")
        self.dedup(keys, stream)
        hs_cache_lookup(self.plan, self.cache, self.cache_capacity, self.unique_keys,
                        self.first_index, -1, self.n_unique, self.topk_score, self.topk_index,
                        self.miss_pos, self.miss_first, self.n_miss, stream=stream)
        hs_scatter(q_req, self.R, self.q_row_bytes, self.miss_first, 0, self.cap, self.n_miss,
                   self.q_miss, stream=stream)
        if score_events is not None:
            score_events[0].record(stream)
        hs_score_partial(self.plan, self.q_miss, -1, self.n_miss, corpus, scale, self.ws,
                         stream=stream)
        if score_events is not None:
            score_events[1].record(stream)
        hs_topk_merge(self.plan, -1, self.n_miss, self.miss_score, self.miss_index, self.ws,
                      stream=stream)
        row = self.k * 4
        hs_scatter(self.miss_score, self.cap, row, self.miss_pos, 0, self.cap, self.n_unique,
                   self.topk_score, stream=stream)
        hs_scatter(self.miss_index, self.cap, row, self.miss_pos, 0, self.cap, self.n_unique,
                   self.topk_index, stream=stream)
        hs_cache_insert(self.plan, self.cache, self.cache_capacity, self.unique_keys,
                        self.miss_pos, -1, self.n_unique, self.topk_score, self.topk_index,
                        stream=stream)
        self.deliver(stream)

    # ------------------------------------------------ ready-queue priorities

    def priority(self, phi, s_hat, heavy=None, alpha=1.0, gamma=1.0, delta=0.0, eps=1e-6,
                 stream=None):
        """Eq. 3 / Eq. 7 priorities of this window's fused nodes (after dedup)
        and their ready-queue order; results in self.phi_fused, self.pi,
        self.order (first n_u entries)."""
        import torch
        dev = self.ws.device
        if not hasattr(self, "order"):
            c1 = max(self.cap, 1)
            self.phi_fused = torch.empty(c1, dtype=torch.float64, device=dev)
            self.pi = torch.empty(c1, dtype=torch.float64, device=dev)
            self.order = torch.empty(c1, dtype=torch.int32, device=dev)
        hs_priority(self.plan, self.inverse, self.first_index, -1, self.n_unique, phi, s_hat,
                    heavy, alpha, gamma, delta, eps, self.phi_fused, self.pi, self.order, self.ws,
                    stream=stream)

    # ------------------------------------------------ micro-batching (Eq. 8)

    def score_chunked(self, corpus, n_unique: int, chunk: int, scale=None, stream=None,
                      events=None):
        """Scores the window's n_unique distinct queries (host count) as
        consecutive sub-batches of at most `chunk` queries, one after the
        other on `stream` (the batch limit B_r of Appendix A; small batches
        finish their queries earlier).  Results land in topk_score/index as
        for one batch.  `events`, if given, is a list that receives one
        (start, end) event pair per sub-batch."""
        import torch
        row_q = self.q_row_bytes
        for b0 in range(0, n_unique, chunk):
            nb = min(chunk, n_unique - b0)
            if events is not None:
                ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                ev[0].record(stream)
            q = self.q_unique.data_ptr() + b0 * row_q
            ts = self.topk_score.data_ptr() + b0 * self.k * 4
            ti = self.topk_index.data_ptr() + b0 * self.k * 4
            hs_score_topk(self.plan, q, nb, None, corpus, scale, ts, ti, self.ws, stream=stream)
            if events is not None:
                ev[1].record(stream)
                events.append(ev)

    def score_split(self, corpus, n_unique: int, parts: int, streams, scale=None):
        """Scores the distinct queries as `parts` near-equal sub-batches, each
        on its own stream with its own workspace (the split k_v of Appendix
        A: sub-batches that may run side by side).  The caller orders the
        streams after the current producer and synchronises them."""
        import torch
        if not hasattr(self, "_split_ws") or len(self._split_ws) < parts:
            self._split_ws = [torch.empty_like(self.ws) for _ in range(parts)]
        row_q = self.q_row_bytes
        base = 0
        for j in range(parts):
            nb = n_unique // parts + (1 if j < n_unique % parts else 0)
            if nb == 0:
                continue
            q = self.q_unique.data_ptr() + base * row_q
            ts = self.topk_score.data_ptr() + base * self.k * 4
            ti = self.topk_index.data_ptr() + base * self.k * 4
            hs_score_topk(self.plan, q, nb, None, corpus, scale, ts, ti, self._split_ws[j],
                          stream=streams[j])
            base += nb



# ---------------------------------------------------------------- one call

def dedup(keys, stream=None):
    """Step 1 alone (Sec. 3.3 (I) signature matching) on a device int64
    tensor of R keys: returns (unique_keys, first_index, counts, inverse),
    the per-group tensors trimmed to the n_u groups.  Reads n_u on the host
    (one synchronisation of `stream`)."""
    import torch
    if keys.dtype != torch.int64 or keys.dim() != 1:
        raise TypeError("keys must be a 1-D int64 tensor")
    R = keys.shape[0]
    dev = keys.device
    stream = stream if stream is not None else torch.cuda.current_stream(dev)
    plan = hs_merge_plan(R, 8, 1, 1, HS_BF16, HS_BF16)
    R1 = max(R, 1)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    uk = torch.empty(R1, dtype=torch.int64, device=dev)
    fi = torch.empty(R1, dtype=torch.int32, device=dev)
    ct = torch.empty(R1, dtype=torch.int32, device=dev)
    inv = torch.empty(R1, dtype=torch.int32, device=dev)
    nu_dev = torch.zeros(1, dtype=torch.int64, device=dev)
    nu = hs_dedup(plan, keys if R else None, uk, fi, ct, inv, nu_dev, True, ws, stream=stream)
    return uk[:nu], fi[:nu], ct[:nu], inv[:R]


def merge_retrieval(keys, q_req, corpus, k: int, scale=None, workflow_offsets=None,
                    max_unique: int = 0, stream=None):
    """The whole window in one call: dedup (Sec. 3.3 (I)), one batched exact
    top-k retrieval per distinct query (Appendix A batching), delivery of each
    group's result to every request (Sec. 3.3 (I)).  keys [R] int64,
    q_req [R x d] (float32 or bfloat16), corpus [N x d] (float32, bfloat16, or
    float8_e4m3fn / uint8 codes with scale [N] float32), all on one device;
    workflow_offsets: host CSR of W + 1 request offsets, or None for one
    workflow.  Returns a dict of device tensors: out_score / out_index
    [R x k] (per request), unique_keys / first_index / counts [n_u],
    inverse [R], topk_score / topk_index [n_u x k], and n_unique (an int:
    the call reads it on the host once) and `retrieval`, the MergedRetrieval
    that owns them (workflow_results(w) gives workflow w's rows)."""
    import torch
    stream = stream if stream is not None else torch.cuda.current_stream(keys.device)
    R, d = q_req.shape
    N = corpus.shape[0]
    offs = None if workflow_offsets is None else [int(x) for x in workflow_offsets]
    W = 1 if offs is None else len(offs) - 1
    m = MergedRetrieval(R, d, N, k, dtype_code(q_req), dtype_code(corpus), device=keys.device,
                        max_unique=max_unique, n_workflows=W, workflow_offsets=offs)
    m.run(keys, q_req, corpus, scale, stream=stream)
    stream.synchronize()
    nu = int(m.n_unique.item())
    return {"out_score": m.out_score[:R], "out_index": m.out_index[:R],
            "unique_keys": m.unique_keys[:nu], "first_index": m.first_index[:nu],
            "counts": m.counts[:nu], "inverse": m.inverse[:R],
            "topk_score": m.topk_score[:nu], "topk_index": m.topk_index[:nu],
            "n_unique": nu, "retrieval": m}
