"""Seeded synthetic workloads for merged retrieval.

Stand-ins for the paper's traffic (its experimental setup: many concurrent
RAG / web-search workflows whose retrieval nodes repeat hot queries following
a Zipf law, over bge-large embeddings held in pgvector).  Neither the datasets
nor the embedding model are available, so requests, query vectors and the
chunk corpus are drawn here from seeded generators:

* request keys: Zipf(s) ranks over M query templates, mapped to template ids
  by a seeded permutation; a request's key is a 64-bit signature-like value
  drawn per template (or, for chunk-embedding dedup, the chunk row id itself);
* vectors: unit-norm Gaussian rows, rounded fp64 -> fp32 -> storage type
  (fp32, bf16, or OCP fp8 e4m3 with a per-row fp32 scale = max|x|/448).

This module holds none of the method's arithmetic and is the only code shared
by the oracle side and the GPU side (it produces the bytes both consume).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsynth.so")
_lib = None

# named streams
S_QUERY, S_CORPUS, S_TABLE, S_ZIPF, S_PERM, S_KEY, S_SLOTS = 1, 2, 3, 4, 5, 6, 7
S_TEXT, S_RENDER = 8, 9
S_SCHED = 10
ENC = {"f32": 0, "bf16": 1, "fp8": 2}
BASE_SEED = 20260722


def build(verbose: bool = False) -> str:
    """Compile libsynth.so with gcc (IEEE semantics, no fast-math)."""
    src = os.path.join(_HERE, "gen.c")
    tmp = _SO + ".tmp"
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-pthread", "-std=c11", src, "-lm", "-o", tmp]
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
    u64, i64, i32, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    lib.syn_stream_base.argtypes = [u64, u64]
    lib.syn_stream_base.restype = u64
    lib.syn_draw.argtypes = [u64, u64]
    lib.syn_draw.restype = u64
    lib.syn_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.syn_f32_to_bf16.restype = ctypes.c_uint16
    lib.syn_e4m3_encode.argtypes = [ctypes.c_double]
    lib.syn_e4m3_encode.restype = ctypes.c_uint8
    lib.syn_gaussian_rows.argtypes = [u64, u64, vp, i64, i64, i64, i32, vp, vp, i32]
    lib.syn_gaussian_rows.restype = i32
    lib.syn_permutation.argtypes = [u64, u64, i64, vp]
    lib.syn_permutation.restype = i32
    lib.syn_zipf_ranks.argtypes = [u64, u64, i64, ctypes.c_double, i64, vp]
    lib.syn_zipf_ranks.restype = i32
    _lib = lib
    return lib


def default_threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def gaussian_rows(seed: int, stream: int, n_rows: int, dim: int, enc: str,
                  first: int = 0, row_ids: Optional[np.ndarray] = None,
                  threads: Optional[int] = None):
    """Rows of a unit-norm Gaussian matrix in storage encoding `enc`.

    Returns (data, scale); scale is None unless enc == 'fp8'.  Row i is
    logical row row_ids[i] (or first + i)."""
    lib = _load()
    if row_ids is not None:
        row_ids = np.ascontiguousarray(row_ids, dtype=np.int64)
        n_rows = int(row_ids.shape[0])
    dt = {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[enc]
    out = np.empty((n_rows, dim), dtype=dt)
    scale = np.empty((n_rows,), dtype=np.float32) if enc == "fp8" else None
    rc = lib.syn_gaussian_rows(seed, stream, _ptr(row_ids), first, n_rows, dim, ENC[enc],
                               _ptr(out), _ptr(scale), threads or default_threads())
    if rc != 0:
        raise ValueError(f"syn_gaussian_rows failed ({rc})")
    return out, scale


def permutation(seed: int, stream: int, m: int) -> np.ndarray:
    out = np.empty((m,), dtype=np.int64)
    if _load().syn_permutation(seed, stream, m, _ptr(out)) != 0:
        raise ValueError("syn_permutation failed")
    return out


def zipf_ranks(seed: int, stream: int, m: int, s: float, n: int) -> np.ndarray:
    out = np.empty((n,), dtype=np.int64)
    if _load().syn_zipf_ranks(seed, stream, m, s, n, _ptr(out)) != 0:
        raise ValueError("syn_zipf_ranks failed")
    return out


def template_keys(seed: int, template_ids: np.ndarray) -> np.ndarray:
    """64-bit signature-like key per template id (full int64 range)."""
    lib = _load()
    base = lib.syn_stream_base(seed, S_KEY)
    ids = np.asarray(template_ids, dtype=np.int64)
    uniq, inv = np.unique(ids, return_inverse=True)
    vals = np.array([lib.syn_draw(base, int(t)) for t in uniq], dtype=np.uint64)
    return vals.view(np.int64)[inv].reshape(ids.shape)


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float32 exactly."""
    return (np.asarray(a, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# workload configurations (sizes of the five benchmark workloads)

@dataclass(frozen=True)
class Config:
    name: str
    n_workflows: int
    per_workflow: int
    n_templates: int          # query templates (or chunk pool for dedup-only)
    zipf_s: float             # 0 => the tiny fixed-sharing layout
    dim: int
    q_enc: str
    c_enc: str
    n_corpus: int
    k: int
    dedup_only: bool = False  # chunk-embedding dedup + row gather, no scoring
    desc: str = ""

    @property
    def n_requests(self) -> int:
        return self.n_workflows * self.per_workflow


CONFIGS = {
    "tiny": Config("tiny", 4, 8, 20, 0.0, 384, "f32", "f32", 4096, 10,
                   desc="4 workflows x 8 queries, 4 shared query ids, d=384 fp32, "
                        "4,096 chunks, k=10"),
    "ridge1m": Config("ridge1m", 64, 32, 512, 1.1, 768, "bf16", "bf16", 1_000_000, 10,
                      desc="64 workflows x 32 queries, Zipf(1.1) over 512 templates, "
                           "d=768 bf16, 1,000,000 chunks bf16, k=10"),
    "dedup256k": Config("dedup256k", 1024, 256, 200_000, 1.0, 1024, "bf16", "bf16",
                        200_000, 0, dedup_only=True,
                        desc="1,024 workflows x 256 chunk ids, Zipf(1.0) over 200,000 "
                             "chunks, gather of d=1024 bf16 rows"),
    "mfma4m": Config("mfma4m", 512, 64, 16_384, 0.8, 1024, "bf16", "bf16", 4_000_000, 32,
                     desc="512 workflows x 64 queries, Zipf(0.8) over 16,384 templates, "
                          "d=1024 bf16, 4,000,000 chunks bf16, k=32"),
    "fp8_20m": Config("fp8_20m", 256, 64, 4_096, 1.1, 768, "bf16", "fp8", 20_000_000, 100,
                      desc="256 workflows x 64 queries, Zipf(1.1) over 4,096 templates, "
                           "d=768, 20,000,000 chunks fp8 e4m3 + fp32 row scale, k=100"),
}
# positional aliases in the order the workloads are listed
ORDER = ["tiny", "ridge1m", "dedup256k", "mfma4m", "fp8_20m"]


@dataclass
class Workload:
    cfg: Config
    seed: int
    keys: np.ndarray                 # int64 [R]
    template_ids: np.ndarray         # int64 [R]
    workflow_offsets: np.ndarray     # int64 [W+1]
    q_req: Optional[np.ndarray]      # [R, d] f32 or bf16 bits
    corpus: Optional[np.ndarray]     # [N, d] f32 / bf16 bits / e4m3 codes
    scale: Optional[np.ndarray]      # [N] f32 (fp8 only)
    table: Optional[np.ndarray] = None   # [pool, d] bf16 bits (dedup-only)
    n_corpus: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def R(self) -> int:
        return int(self.keys.shape[0])

    @property
    def dim(self) -> int:
        return self.cfg.dim

    @property
    def k(self) -> int:
        return self.cfg.k


def request_template_ids(cfg: Config, seed: int) -> np.ndarray:
    R = cfg.n_requests
    if cfg.zipf_s == 0.0:
        # tiny layout: each workflow has 4 shared ids (0..3) and 4 private ids;
        # slot order shuffled per workflow
        assert cfg.per_workflow == 8
        rows = []
        for w in range(cfg.n_workflows):
            ids = np.array([0, 1, 2, 3] + [4 + 4 * w + j for j in range(4)], dtype=np.int64)
            p = permutation(seed, S_SLOTS * 1000 + w, 8)
            rows.append(ids[p])
        return np.concatenate(rows)
    ranks = zipf_ranks(seed, S_ZIPF, cfg.n_templates, cfg.zipf_s, R)
    perm = permutation(seed, S_PERM, cfg.n_templates)
    return perm[ranks]


def make(name: str, seed: Optional[int] = None, n_corpus: Optional[int] = None,
         with_corpus: bool = True, threads: Optional[int] = None) -> Workload:
    """Build a workload.  `n_corpus` overrides the corpus size (smaller test
    variants of the same shape); `with_corpus=False` skips the corpus."""
    cfg = CONFIGS[name]
    if seed is None:
        seed = BASE_SEED + ORDER.index(name)
    W, Qw = cfg.n_workflows, cfg.per_workflow
    offsets = np.arange(W + 1, dtype=np.int64) * Qw
    tids = request_template_ids(cfg, seed)
    if cfg.dedup_only:
        keys = tids.copy()       # chunk row ids index the embedding table
        pool = cfg.n_templates if n_corpus is None else n_corpus
        if n_corpus is not None:
            keys = keys % pool
        table = None
        if with_corpus:
            table, _ = gaussian_rows(seed, S_TABLE, pool, cfg.dim, "bf16", threads=threads)
        return Workload(cfg, seed, keys, tids, offsets, None, None, None, table=table,
                        n_corpus=pool)
    keys = template_keys(seed, tids)
    q_req, _ = gaussian_rows(seed, S_QUERY, 0, cfg.dim, cfg.q_enc, row_ids=tids,
                             threads=threads)
    N = cfg.n_corpus if n_corpus is None else int(n_corpus)
    corpus = scale = None
    if with_corpus:
        corpus, scale = gaussian_rows(seed, S_CORPUS, N, cfg.dim, cfg.c_enc, threads=threads)
    return Workload(cfg, seed, keys, tids, offsets, q_req, corpus, scale, n_corpus=N)


def expected_unique(cfg: Config) -> float:
    """E[number of distinct templates] = sum_r 1 - (1 - p_r)^R (Zipf configs)."""
    r = np.arange(1, cfg.n_templates + 1, dtype=np.float64)
    p = r ** (-cfg.zipf_s)
    p /= p.sum()
    return float(np.sum(1.0 - (1.0 - p) ** cfg.n_requests))


def window_stream(name: str, n_windows: int, seed: Optional[int] = None,
                  threads: Optional[int] = None) -> list:
    """Successive merge windows of one workload's traffic: each window draws
    its own Zipf sample of template ids (stream S_ZIPF * 1000 + w) over the
    same templates, so hot templates recur across windows with the same key
    and query row.  Returns one Workload per window, without a corpus."""
    cfg = CONFIGS[name]
    if cfg.dedup_only or cfg.zipf_s == 0.0:
        raise ValueError(f"{name}: window streams need a Zipf retrieval workload")
    if seed is None:
        seed = BASE_SEED + ORDER.index(name)
    perm = permutation(seed, S_PERM, cfg.n_templates)
    offsets = np.arange(cfg.n_workflows + 1, dtype=np.int64) * cfg.per_workflow
    out = []
    for w in range(n_windows):
        ranks = zipf_ranks(seed, S_ZIPF * 1000 + w, cfg.n_templates, cfg.zipf_s,
                           cfg.n_requests)
        tids = perm[ranks]
        keys = template_keys(seed, tids)
        q_req, _ = gaussian_rows(seed, S_QUERY, 0, cfg.dim, cfg.q_enc, row_ids=tids,
                                 threads=threads)
        out.append(Workload(cfg, seed, keys, tids, offsets, q_req, None, None,
                            n_corpus=cfg.n_corpus, extra={"window": w}))
    return out


# --------------------------------------------------------------------------
# node texts (inputs of the signature step)

_WS = b" \t\n\r\x0b\x0c"
_ACCENTED = ["\u00e9", "\u00c9", "\u00fc", "\u00df", "\u4e2d"]   # multi-byte UTF-8


def template_text(seed: int, template_id: int) -> bytes:
    """Canonical text of a query template: 4-15 pseudo-words of 2-10 lower-case
    letters (some carrying a multi-byte UTF-8 letter), single spaces."""
    g = np.random.default_rng([seed, S_TEXT, int(template_id)])
    words = []
    for _ in range(int(g.integers(4, 16))):
        w = "".join(chr(97 + int(c)) for c in g.integers(0, 26, size=int(g.integers(2, 11))))
        if g.random() < 0.05:
            w += _ACCENTED[int(g.integers(0, len(_ACCENTED)))]
        words.append(w)
    return " ".join(words).encode("utf-8")


def render_texts(seed: int, template_ids: np.ndarray, vary: bool = True):
    """Request texts packed back to back: (uint8 buffer, int64 offsets [R+1]).
    With `vary`, each request renders its template with its own case flips of
    ASCII letters and runs of ASCII whitespace between, before and after the
    words, as users type the same query differently; the normalised forms of
    a template's renderings are identical."""
    parts = []
    cache = {}
    for i, t in enumerate(np.asarray(template_ids, dtype=np.int64)):
        t = int(t)
        if t not in cache:
            cache[t] = template_text(seed, t)
        base = cache[t]
        if not vary:
            parts.append(base)
            continue
        g = np.random.default_rng([seed, S_RENDER, i])
        out = bytearray()
        if g.random() < 0.3:
            out += bytes(_WS[int(c)] for c in g.integers(0, 6, size=int(g.integers(1, 4))))
        for j, word in enumerate(base.split(b" ")):
            if j:
                n = int(g.integers(1, 4)) if g.random() < 0.3 else 1
                out += bytes(_WS[int(c)] for c in g.integers(0, 6, size=n)) if n > 1 or \
                    g.random() < 0.2 else b" "
            flips = g.random(len(word)) < 0.15
            out += bytes((c - 32) if (f and 97 <= c <= 122) else c for c, f in zip(word, flips))
        if g.random() < 0.3:
            out += bytes(_WS[int(c)] for c in g.integers(0, 6, size=int(g.integers(1, 4))))
        parts.append(bytes(out))
    off = np.zeros(len(parts) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in parts])
    buf = np.frombuffer(b"".join(parts), dtype=np.uint8).copy()
    return buf, off


def scheduler_inputs(w: Workload):
    """Per-request scheduler state for the priority step: phi (fp32, a mix of
    a few repeated values -- so that fused sums tie -- and continuous values
    in [0, 50)), the remaining-time estimate of each request's workflow
    (fp32 in [0.1, 20), shared by the workflow's requests) and a heavy flag
    per workflow (about 15 % of workflows)."""
    g = np.random.default_rng([w.seed, S_SCHED])
    R = w.R
    n_wf = len(w.workflow_offsets) - 1
    wf = np.repeat(np.arange(n_wf), np.diff(w.workflow_offsets))
    discrete = np.array([0.5, 1.0, 2.0, 4.0], dtype=np.float32)[g.integers(0, 4, size=R)]
    cont = (g.random(R) * 50).astype(np.float32)
    phi = np.where(g.random(R) < 0.5, discrete, cont).astype(np.float32)
    s_wf = (0.1 + g.random(n_wf) * 19.9).astype(np.float32)
    heavy_wf = (g.random(n_wf) < 0.15).astype(np.uint8)
    return phi, s_wf[wf], heavy_wf[wf]

