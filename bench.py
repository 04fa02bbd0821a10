#!/usr/bin/env python3
"""Benchmark of the merged-retrieval hot path on one MI355X.

One step = one merge window of the whole path on the device: dedup of the
request signatures, gather of the representative query rows, exact bf16 MFMA
scoring + top-k of the distinct queries against the HBM-resident corpus, and
delivery of every result to each request.  Inputs are synthetic (seeded) and
resident in HBM before timing starts; the distinct count stays on the device
(no host synchronisation inside a step).

Default workload (the largest single-GPU one, compute-bound): 512 workflows
x 64 retrieval queries, query ids Zipf(0.8) over 16,384 templates (about
10,000 distinct), d=1024 bf16 unit-norm, 4,000,000-chunk bf16 corpus, k=32.

Prints ONE JSON line.  `value` = logical requests per second of the timed
steps.  `roofline` describes the dominant kernel (the scoring kernel), timed
with HIP events on its own stream inside the timed region.  `cpu_baseline`
times the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "merged retrieval queries/s + achieved HBM GB/s or MFMA % (dedup+score+top-k)"
PEAK_HBM_GBS = 8000.0
PEAK_MFMA = {"bf16": 2500.0}          # dense TFLOP/s (no sparsity)
PEAK_FP32_VECTOR = 157.3              # TFLOP/s, fp32 on the vector units
DEFAULT_WORKLOAD = "mfma4m"


def traffic_file(workload: str) -> str:
    """Committed HBM counter summary of the score step on one workload."""
    return os.path.join(ROOT, "profiles", f"score_step_{workload}_traffic.json")


KERNEL_SOURCES = ["paper_2607_22578_amd/csrc/score_mfma.hip", "paper_2607_22578_amd/csrc/score.hip",
                  "paper_2607_22578_amd/csrc/common.h"]
# The score step (hs_score_partial) is four launches on one stream: the query
# tiling, the seed pass, the seed selection (which also restarts the shared
# thresholds) and the main pass.  Its HIP-event duration is the sum of those
# kernels' durations.
EV_EVERY = 4
SCORE_STEP = ("score step = tile_queries_kernel + score_mfma_dma (seed pass) + mfma_seed_kernel "
              "+ score_mfma_dma (main pass)")
SCORE_STEP_VALU = "score step = score_partial_valu (fp32, vector units)"


DEDUP_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "dedup_gather_dedup256k_traffic.json")
DEDUP_SOURCES = ["paper_2607_22578_amd/csrc/dedup.hip", "paper_2607_22578_amd/csrc/gather.hip",
                 "paper_2607_22578_amd/csrc/common.h"]


def kernel_source_hash(sources=None) -> str:
    """Hash of the kernels' code (the score kernels by default) with comments
    and blank lines removed, so that a change of comments alone keeps the
    counters that were taken."""
    h = hashlib.sha256()
    for p in (KERNEL_SOURCES if sources is None else sources):
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    help="mfma4m (default), ridge1m, fp8_20m, tiny or dedup256k")
    ap.add_argument("--seed", type=int, default=None,
                    help="base seed of the synthetic workload (default: 20260722 + the "
                         "workload's position in the list tiny, ridge1m, dedup256k, mfma4m, "
                         "fp8_20m)")
    ap.add_argument("--raw-ids", action="store_true",
                    help="key-range ablation: request keys are the small template ids "
                         "themselves instead of 64-bit signature-like values (the dedup may "
                         "then take its direct-addressing path; the line reports the path)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="distinct queries scored by the oracle for the CPU baseline (default: "
                         "as many as take about 20 s on the oracle's threads)")
    ap.add_argument("--oracle-threads", type=int, default=0,
                    help="threads of the CPU baseline (default: OMP_NUM_THREADS if set, else "
                         "the CPUs this process may run on)")
    ap.add_argument("--no-merge", action="store_true",
                    help="ablation: every request is scored on its own (no dedup merge)")
    ap.add_argument("--corpus-rows", type=int, default=0,
                    help="override the corpus size (e.g. one GPU's shard of a sharded corpus)")
    ap.add_argument("--reuse-store", type=int, default=0,
                    help="cross-window reuse: a result store of this many entries (a power "
                         "of two); each step is the next window of the workload's request "
                         "stream, scored only where the store misses")
    ap.add_argument("--signatures", action="store_true",
                    help="each step starts from node descriptions: the request keys are the "
                         "SHA-256 signatures of the requests' texts (hs_signature), not "
                         "precomputed")
    ap.add_argument("--sig-nodes", type=int, default=0,
                    help="only time hs_signature on this many request nodes of the workload's "
                         "traffic (one JSON line of its own)")
    ap.add_argument("--priorities", action="store_true",
                    help="each step also computes the fused nodes' priorities and ready-queue "
                         "order (hs_priority) after the dedup")
    ap.add_argument("--prio-only", default="",
                    help="only time hs_dedup + hs_priority on this workload's requests (e.g. "
                         "dedup256k; one JSON line of its own)")
    ap.add_argument("--batch-curve", action="store_true",
                    help="micro-batching (Eq. 8): score latency against batch size, and the "
                         "window's distinct queries scored in sub-batches of at most B or split "
                         "over k streams (mean / max completion); one JSON line of its own")
    ap.add_argument("--batch-sizes", type=str, default=None,
                    help="with --batch-curve: only the latency curve, at these comma-separated "
                         "batch sizes (default: the full curve 1,2,4,...,2048 and the sub-batch "
                         "and stream-split runs)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one window (dedup, gather, score, merge, delivery) as a HIP "
                         "graph after the warm-up and time its replays (the score-step events "
                         "then come from eager steps after the timed region)")
    ap.add_argument("--corpus-layout", choices=("tiled", "rows"), default="tiled",
                    help="storage of a BF16/FP8 corpus: tiled (default; hs_tile_corpus, made "
                         "once before the warm-up, as an index is) or row-major (rows); an "
                         "F32 corpus is always row-major")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (counter calibration)")
    return ap.parse_args()


def copy_calibration(nbytes: int):
    import torch
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "launches": 5}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU; the multi-GPU (corpus-sharded) path is a "
              "design only, so --gpus must be 1", file=sys.stderr)
        sys.exit(2)
    if args.copy_bytes:
        copy_calibration(args.copy_bytes)
        return
    if args.sig_nodes:
        signature_bench(args)
        return
    if args.prio_only:
        priority_bench(args)
        return
    if args.batch_curve:
        batch_curve_bench(args)
        return
    if args.workload == "dedup256k":
        dedup_bench(args)
        return

    import numpy as np
    import torch

    import paper_2607_22578_amd as hs
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.time()
    w = synth.make(args.workload, seed=args.seed, n_corpus=args.corpus_rows or None)
    t_gen = time.time() - t_gen
    if args.raw_ids:
        if args.no_merge:
            raise SystemExit("--raw-ids and --no-merge exclude each other")
        # the template id itself as the key: same groups, small key range
        w.keys = w.template_ids.astype(np.int64).copy()
    if args.no_merge:
        # every request its own key: the same rows and corpus, scored unmerged
        w.keys = np.arange(w.R, dtype=np.int64)
    cfg = w.cfg
    R, d, N, k = w.R, w.dim, w.n_corpus, w.k
    enc = {"f32": hs.HS_F32, "bf16": hs.HS_BF16, "fp8": hs.HS_FP8_E4M3}
    qdt, cdt = enc[cfg.q_enc], enc[cfg.c_enc]
    f32 = cfg.c_enc == "f32"

    def to_dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    keys, q_req, corpus = to_dev(w.keys), to_dev(w.q_req), to_dev(w.corpus)
    scale = to_dev(w.scale) if w.scale is not None else None
    tiled = args.corpus_layout == "tiled" and not f32
    m = hs.MergedRetrieval(R, d, N, k, qdt, cdt, device=dev, tiled_corpus=tiled)
    stream = torch.cuda.Stream(dev)   # default priority
    if tiled:
        # the corpus is the retrieval index: laid out once, before any timing
        corpus = m.tile_corpus(corpus, stream)
        torch.cuda.synchronize(dev)
    sig = None
    if args.signatures:
        if args.no_merge:
            raise SystemExit("--signatures and --no-merge exclude each other")
        buf, off = synth.render_texts(w.seed, w.template_ids)
        sig = SigInputs(hs, dev, buf, off, k)
        keys = sig.keys
    sig_ev = {}
    prio = None
    if args.priorities:
        phi_h, s_h, y_h = synth.scheduler_inputs(w)
        prio = (to_dev(phi_h), to_dev(s_h), to_dev(y_h))
    prio_ev = {}
    windows = None
    if args.reuse_store:
        # successive windows of the same traffic: window i is step i of the run
        windows = [(to_dev(x.keys), to_dev(x.q_req))
                   for x in synth.window_stream(args.workload, args.warmup + args.steps)]
        m.enable_cache(args.reuse_store, stream)
    step_no = [0]

    def step(ev=None):
        if sig is not None:
            if ev is not None:
                sig_ev[id(ev)][0].record(stream)
            sig.run(stream)
            if ev is not None:
                sig_ev[id(ev)][1].record(stream)
        if windows is not None:
            wk, wq = windows[step_no[0]]
            step_no[0] += 1
            m.run_cached(wk, wq, corpus, scale, stream, score_events=ev)
            return
        m.dedup(keys, stream)
        if prio is not None:
            if ev is not None:
                prio_ev[id(ev)][0].record(stream)
            m.priority(*prio, **PRIO_WEIGHTS, stream=stream)
            if ev is not None:
                prio_ev[id(ev)][1].record(stream)
        m.gather_queries(q_req, stream)
        if ev is not None:
            ev[0].record(stream)
        m.score_partial(corpus, scale, -1, stream)
        if ev is not None:
            ev[1].record(stream)
        m.topk_merge(-1, stream)
        m.deliver(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    n_u = int(m.n_unique.item())
    graph = None
    if args.graph:
        if sig is not None or prio is not None or windows is not None:
            raise SystemExit("--graph captures the plain window (no --signatures, "
                             "--priorities or --reuse-store)")
        # the window issues kernel launches only (device-side distinct count)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            step()
        torch.cuda.synchronize(dev)

    # The score step is timed with HIP events on its stream inside the timed
    # region, on every EV_EVERY-th step: each timing event costs the stream
    # a few microseconds, so fewer of them disturb the throughput less.
    ev_steps = list(range(0, args.steps, EV_EVERY))
    evs = {i: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for i in ev_steps}
    for e in evs.values():
        sig_ev[id(e)] = (torch.cuda.Event(enable_timing=True),
                         torch.cuda.Event(enable_timing=True))
        prio_ev[id(e)] = (torch.cuda.Event(enable_timing=True),
                          torch.cuda.Event(enable_timing=True))
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    wall0 = time.perf_counter()
    t_start.record(stream)
    if graph is not None:
        with torch.cuda.stream(stream):
            for i in range(args.steps):
                graph.replay()
    else:
        for i in range(args.steps):
            step(evs.get(i))
    t_end.record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps
    if graph is not None:   # score-step events from eager steps (outside the timed region)
        for i in ev_steps:
            step(evs[i])
        torch.cuda.synchronize(dev)
    kern_samples = np.array([a.elapsed_time(b) for a, b in evs.values()])
    kern_ms = float(np.mean(kern_samples))

    reuse = None
    if windows is not None:
        # replay from an empty store (deterministic), reading each window's
        # distinct and miss counts; the timed steps are windows warmup.. on
        hs.hs_cache_reset(m.plan, m.cache, m.cache_capacity, stream=stream)
        nus, nms = [], []
        for wk, wq in windows:
            m.run_cached(wk, wq, corpus, scale, stream)
            torch.cuda.synchronize(dev)
            nus.append(int(m.n_unique.item()))
            nms.append(int(m.n_miss.item()))
        nus, nms = np.array(nus[args.warmup:]), np.array(nms[args.warmup:])
        reuse = {"capacity": args.reuse_store, "store_bytes": int(m.cache.numel()),
                 "windows": len(windows), "mean_unique": round(float(nus.mean()), 2),
                 "mean_miss": round(float(nms.mean()), 2),
                 "hit_frac": round(1.0 - float(nms.sum()) / max(int(nus.sum()), 1), 4)}
        n_u = float(nms.mean())   # queries the score step processes per window
        n_distinct = float(nus.mean())
        # the windows whose score steps the events timed: a window whose keys
        # all hit the store scores nothing and moves no corpus bytes
        timed_miss = nms[np.array(ev_steps)]
        reuse_pricing = (float(timed_miss.mean()), float((timed_miss > 0).mean()))
    else:
        n_distinct = n_u
        reuse_pricing = None

    # stage breakdown (separate, untimed-for-value pass)
    st_ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    reps = 0 if windows is not None else 10
    acc = np.zeros(5)
    for _ in range(reps):
        st_ev[0].record(stream)
        m.dedup(keys, stream)
        st_ev[1].record(stream)
        m.gather_queries(q_req, stream)
        st_ev[2].record(stream)
        m.score_partial(corpus, scale, -1, stream)
        st_ev[3].record(stream)
        m.topk_merge(-1, stream)
        st_ev[4].record(stream)
        m.deliver(stream)
        st_ev[5].record(stream)
        torch.cuda.synchronize(dev)
        acc += [st_ev[i].elapsed_time(st_ev[i + 1]) for i in range(5)]
    sig_stats = None
    if sig is not None:
        sig_ms = float(np.mean([sig_ev[id(e)][0].elapsed_time(sig_ev[id(e)][1])
                                for e in evs.values()]))
        sig_stats = sig.stats(sig_ms)
    prio_stats = None
    if prio is not None:
        pms = float(np.mean([prio_ev[id(e)][0].elapsed_time(prio_ev[id(e)][1])
                             for e in evs.values()]))
        prio_stats = {"kernels": "priority_clear/sum/pi/chunk_sort/merge/order",
                      "n_requests": R, "n_unique": n_u, "ms": round(pms, 4)}
    stages = dict(zip(["dedup", "gather", "score_partial", "topk_merge", "deliver"],
                      (acc / max(reps, 1)).round(4).tolist())) if reps else None

    # roofline of the scoring kernel: algorithmic work per launch
    c_bytes = N * d * {"fp8": 1, "bf16": 2, "f32": 4}[cfg.c_enc] + \
        (N * 4 if cfg.c_enc == "fp8" else 0)
    n_q = n_u
    if reuse_pricing is not None:   # mean over the timed windows
        n_q, scored = reuse_pricing
        c_bytes *= scored
    q_bytes = n_q * d * (4 if f32 else 2)
    alg_bytes = c_bytes + q_bytes
    alg_flops = 2.0 * n_q * N * d
    t_s = kern_ms * 1e-3
    tflops = alg_flops / t_s / 1e12
    gbs = alg_bytes / t_s / 1e9
    t_mfma = alg_flops / (PEAK_MFMA["bf16"] * 1e12)
    t_hbm = alg_bytes / (PEAK_HBM_GBS * 1e9)
    t_alu = alg_flops / (PEAK_FP32_VECTOR * 1e12)
    if f32 and t_alu >= t_hbm:   # fp32 inputs run on the vector units
        roof = {"bound": "alu", "achieved": round(tflops, 3), "peak": PEAK_FP32_VECTOR,
                "unit": "TFLOP/s", "frac": round(tflops / PEAK_FP32_VECTOR, 4)}
    elif f32:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}
    elif t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_MFMA["bf16"],
                "unit": "TFLOP/s", "frac": round(tflops / PEAK_MFMA["bf16"], 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}
    roof["traffic"] = None
    roof["kernel"] = SCORE_STEP_VALU if f32 else SCORE_STEP
    roof["kernel_ms"] = round(kern_ms, 4)
    roof["kernel_ms_p10_p50_p90"] = [round(float(np.percentile(kern_samples, p)), 4)
                                     for p in (10, 50, 90)]
    roof["algorithmic_bytes"] = alg_bytes
    roof["algorithmic_flops"] = alg_flops
    roof["hbm_gbs_algorithmic"] = round(gbs, 1)
    roof["hbm_frac_algorithmic"] = round(gbs / PEAK_HBM_GBS, 4)
    roof["mfma_frac"] = round(tflops / PEAK_MFMA["bf16"], 4)
    src_hash = kernel_source_hash()
    roof["kernel_source"] = src_hash
    if windows is not None:
        roof["note"] = ("reuse mode: score-step work priced over the timed windows (their mean "
                        "miss count; corpus bytes only where a window has a miss)")
    tf = traffic_file(args.workload)
    if not (args.no_merge or args.raw_ids or args.corpus_rows or windows is not None
            or args.seed is not None or (args.corpus_layout == "rows" and not f32)) \
            and os.path.exists(tf):
        tr = json.load(open(tf))
        if tr.get("kernel_source") == src_hash:
            roof["traffic"] = tr.get("hbm_bytes_per_launch")
            # bytes beyond L2 (counters) per second of the timed score step
            roof["traffic_gbs"] = round(roof["traffic"] / t_s / 1e9, 1)

    value = R * args.steps / (total_ms * 1e-3)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if f32 else "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.desc}", "n_requests": R, "n_unique": n_distinct,
                   "dim": d, "n_corpus": N, "k": k, "query_dtype": cfg.q_enc,
                   "corpus_dtype": cfg.c_enc, "seed": w.seed,
                   "merge": not args.no_merge, "reuse": reuse,
                   "signatures": args.signatures, "priorities": args.priorities,
                   "raw_ids": args.raw_ids, "dedup_path": dedup_path(w.keys),
                   "graph": args.graph, "corpus_layout": "tiled" if tiled else "rows"},
        "unique_queries_per_s": round(n_distinct * args.steps / (total_ms * 1e-3), 1),
        "stages_ms": stages,
        "wall_s_timed": round(wall, 4),
        "roofline": roof,
    }
    if sig_stats is not None:
        out["signature_step"] = sig_stats
    if prio_stats is not None:
        out["priority_step"] = prio_stats

    if not args.no_cpu_baseline and windows is None:
        out["cpu_baseline"] = cpu_baseline(w, n_u, args.cpu_sample, args.oracle_threads)
    print(json.dumps(out), flush=True)


# SHA-256 work per 64-byte block, counted from the FIPS 180-4 definitions:
# 64 rounds of 26 operations (T1: Sigma1 5, Ch 4, 4 additions; T2: Sigma0 5,
# Maj 5, 1 addition; e and a: 2 additions), 48 schedule words of 13 (two sigma
# functions of 5, 3 additions) and 8 final additions.
SHA_OPS_PER_BLOCK = 64 * 26 + 48 * 13 + 8
# 32-bit integer VALU peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
PEAK_INT32_OPS = 256 * 4 * 16 * 2.4e9


def _normalised_len(t: bytes) -> int:
    return len(b" ".join(t.lower().split()))


class SigInputs:
    """Device buffers of one window's request nodes for hs_signature:
    retrieval nodes (operator type 2) with Top-K as their parameter bytes and
    their query text, normalised; no predecessors."""

    def __init__(self, hs, dev, buf, off, k):
        import numpy as np
        import torch
        self.hs = hs
        n = len(off) - 1
        self.n = n
        self.op = torch.full((n,), 2, dtype=torch.int32, device=dev)
        self.par = torch.from_numpy(np.full(n, k, dtype=np.uint32).view(np.uint8).copy()).to(dev)
        self.poff = torch.arange(0, 4 * (n + 1), 4, dtype=torch.int64, device=dev)
        self.text = torch.from_numpy(buf if buf.size else np.zeros(1, np.uint8)).to(dev)
        self.text_bytes = int(buf.size)
        self.toff = torch.from_numpy(off).to(dev)
        self.digest = torch.empty((max(n, 1), 32), dtype=torch.uint8, device=dev)
        self.keys = torch.empty(max(n, 1), dtype=torch.int64, device=dev)
        raw = buf.tobytes()
        lens = [16 + 4 + _normalised_len(raw[off[i]:off[i + 1]]) for i in range(n)]
        self.blocks = int(sum((L + 8) // 64 + 1 for L in lens))
        self.msg_bytes = int(sum(lens))

    def run(self, stream):
        self.hs.hs_signature(self.op, self.n, 0, self.n, self.digest, self.keys, params=self.par,
                             param_off=self.poff, text=self.text, text_off=self.toff,
                             text_bytes=self.text_bytes, flags=self.hs.HS_SIG_NORMALIZE_TEXT,
                             stream=stream)

    def stats(self, ms: float) -> dict:
        ops = self.blocks * SHA_OPS_PER_BLOCK
        t = ms * 1e-3
        return {"kernel": "signature_kernel", "nodes": self.n, "text_bytes": self.text_bytes,
                "message_bytes": self.msg_bytes, "sha256_blocks": self.blocks,
                "kernel_ms": round(ms, 4), "nodes_per_s": round(self.n / t, 1),
                "roofline": {"bound": "alu", "achieved": round(ops / t / 1e12, 4),
                             "peak": PEAK_INT32_OPS / 1e12, "unit": "Tops/s",
                             "frac": round(ops / t / PEAK_INT32_OPS, 4),
                             "ops_per_block": SHA_OPS_PER_BLOCK}}


def signature_bench(args):
    """hs_signature alone on `--sig-nodes` request nodes drawn like the
    workload's requests (Zipf template ids, per-request renderings)."""
    import numpy as np
    import torch

    import paper_2607_22578_amd as hs
    import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[args.workload]
    seed = synth.BASE_SEED + synth.ORDER.index(args.workload)
    ranks = synth.zipf_ranks(seed, synth.S_ZIPF, cfg.n_templates, cfg.zipf_s, args.sig_nodes)
    tids = synth.permutation(seed, synth.S_PERM, cfg.n_templates)[ranks]
    buf, off = synth.render_texts(seed, tids)
    sig = SigInputs(hs, dev, buf, off, max(cfg.k, 1))
    stream = torch.cuda.Stream(dev)
    for _ in range(args.warmup):
        sig.run(stream)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    a.record(stream)
    for _ in range(args.steps):
        sig.run(stream)
    b.record(stream)
    torch.cuda.synchronize(dev)
    ms = a.elapsed_time(b) / args.steps
    st = sig.stats(ms)
    out = {"metric": "node signatures/s (SHA-256 of Eq. 2 messages)", "value": st["nodes_per_s"],
           "unit": "nodes/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "u32", "data": "synthetic",
           "config": {"workload": f"{args.sig_nodes} request nodes of {cfg.name}'s traffic "
                                  f"(Zipf({cfg.zipf_s}) over {cfg.n_templates} templates), "
                                  "normalised query text + Top-K parameter"},
           "roofline": st["roofline"], "signature_step": st}
    print(json.dumps(out), flush=True)


def dedup_bench(args):
    """The chunk-embedding dedup workload: one step = hs_dedup of the R chunk
    ids of all workflows + the gather of the distinct ids' embedding rows
    (a1 + a2'); value = chunk ids per second."""
    import numpy as np
    import torch

    import paper_2607_22578_amd as hs
    import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.make(args.workload, seed=args.seed)
    R, d = w.R, w.dim
    rows = w.table.shape[0]
    plan = hs.hs_merge_plan(R, d, rows, 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    kd = torch.from_numpy(w.keys).to(dev)
    table = torch.from_numpy(w.table.view(np.int16)).view(torch.bfloat16).to(dev)
    uk = torch.empty(R, dtype=torch.int64, device=dev)
    fi = torch.empty(R, dtype=torch.int32, device=dev)
    ct = torch.empty(R, dtype=torch.int32, device=dev)
    inv = torch.empty(R, dtype=torch.int32, device=dev)
    nu = torch.zeros(1, dtype=torch.int64, device=dev)
    emb = torch.empty((R, d), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.Stream(dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        hs.hs_dedup(plan, kd, uk, fi, ct, inv, nu, None, ws, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        hs.hs_scatter(table, rows, d * 2, uk, 1, R, nu, emb, stream=stream)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    n_u = int(nu.item())
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3))
           for _ in range(0, args.steps, EV_EVERY)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    t0.record(stream)
    for i in range(args.steps):
        step(evs[i // EV_EVERY] if i % EV_EVERY == 0 else None)
    t1.record(stream)
    torch.cuda.synchronize(dev)
    total = t0.elapsed_time(t1)
    dd = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    gg = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    # algorithmic bytes: keys in; distinct keys, survivors, counts and the
    # request map out; the distinct rows read and written once
    alg = R * 8 + n_u * (8 + 4 + 4) + R * 4 + 2 * n_u * d * 2
    t = (dd + gg) * 1e-3
    out = {"metric": "chunk ids/s through dedup + embedding-row gather", "unit": "chunk ids/s",
           "value": round(R * args.steps / (total * 1e-3), 1), "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(total / args.steps, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
           "config": {"workload": f"{w.cfg.name}: {w.cfg.desc}", "n_requests": R,
                      "n_unique": n_u, "dim": d, "table_rows": rows},
           "stages_ms": {"dedup": round(dd, 4), "gather": round(gg, 4)},
           "roofline": {"bound": "hbm", "achieved": round(alg / t / 1e9, 1),
                        "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(alg / t / 1e9 / PEAK_HBM_GBS, 4), "traffic": None,
                        "kernel": "hs_dedup + gather_rows_kernel",
                        "algorithmic_bytes": alg, "kernel_ms": round(dd + gg, 4),
                        "kernel_source": kernel_source_hash(DEDUP_SOURCES)}}
    if os.path.exists(DEDUP_TRAFFIC_FILE):
        tr = json.load(open(DEDUP_TRAFFIC_FILE))
        if tr.get("kernel_source") == out["roofline"]["kernel_source"]:
            out["roofline"]["traffic"] = tr.get("hbm_bytes_per_step")
            out["roofline"]["traffic_gbs"] = round(out["roofline"]["traffic"] / t / 1e9, 1)
    print(json.dumps(out), flush=True)


def batch_curve_bench(args):
    """Latency of the score step (hs_score_topk) against the number of
    queries in one batch, and the window's distinct queries as sequential
    sub-batches of at most B queries (B_r) or as k sub-batches on k streams
    (k_v), with the mean and the largest query completion time (the two terms
    of Eq. 8's objective)."""
    import numpy as np
    import torch

    import paper_2607_22578_amd as hs
    import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.make(args.workload, seed=args.seed)
    cfg = w.cfg
    R, d, N, k = w.R, w.dim, w.n_corpus, w.k
    cdt = {"bf16": hs.HS_BF16, "fp8": hs.HS_FP8_E4M3}[cfg.c_enc]

    def to_dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    keys, q_req, corpus = to_dev(w.keys), to_dev(w.q_req), to_dev(w.corpus)
    scale = to_dev(w.scale) if w.scale is not None else None
    tiled = args.corpus_layout == "tiled"
    m = hs.MergedRetrieval(R, d, N, k, hs.HS_BF16, cdt, device=dev, tiled_corpus=tiled)
    stream = torch.cuda.Stream(dev)
    if tiled:
        corpus = m.tile_corpus(corpus, stream)
        torch.cuda.synchronize(dev)
    nu = m.dedup(keys, stream, host_count=True)
    reps = max(3, min(args.steps, 20))

    def timed(fn):
        out = []
        for r in range(reps + 2):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize(dev)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize(dev)
            if r >= 2:
                out.append(a.elapsed_time(b))
        return float(np.median(out))

    # latency against batch size: the first b request rows as the batch
    m.q_unique[:R].copy_(q_req)
    torch.cuda.synchronize(dev)
    curve = []
    sizes = ([int(x) for x in args.batch_sizes.split(",") if x.strip()] if args.batch_sizes
             else [1, 2, 4, 8, 16, 32, 64, 96, 128, 160, 256, 384, 512, 1024, 2048])
    for b in sizes:
        if b > R:
            break
        ms = timed(lambda: hs.hs_score_topk(m.plan, m.q_unique, b, None, corpus, scale,
                                            m.topk_score, m.topk_index, m.ws, stream=stream))
        curve.append({"batch": b, "ms": round(ms, 4), "queries_per_s": round(b / ms * 1e3, 1)})

    if args.batch_sizes:   # the latency curve alone
        worst = max(curve, key=lambda c: c["ms"])
        out = {"metric": "score latency vs batch size (Eq. 8, Appendix A batch limit)",
               "value": round(worst["batch"] / worst["ms"] * 1e3, 1), "unit": "queries/s",
               "n_gpus": 1, "steps": reps, "warmup": 2, "ms_per_step": worst["ms"],
               "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
               "dtype": "bf16", "data": "synthetic",
               "config": {"workload": f"{cfg.name}: {cfg.desc}", "k": k, "n_corpus": N,
                          "corpus_layout": "tiled" if tiled else "rows"},
               "latency_curve": curve}
        print(json.dumps(out), flush=True)
        return

    # the window's distinct queries in sub-batches of at most B, one after another
    m.gather_queries(q_req, stream)
    torch.cuda.synchronize(dev)
    chunked = []
    for B in sorted({16, 32, 64, 128, 256, nu}):
        if B > nu:
            continue
        runs = []
        for r in range(reps):
            evs = []
            m.score_chunked(corpus, nu, B, scale, stream, events=evs)
            torch.cuda.synchronize(dev)
            t0 = evs[0][0]
            done = [t0.elapsed_time(e[1]) for e in evs]
            sizes = [min(B, nu - j * B) for j in range(len(evs))]
            mean_c = sum(c * s for c, s in zip(done, sizes)) / nu
            runs.append((mean_c, done[-1]))
        mean_c = float(np.median([x[0] for x in runs]))
        max_c = float(np.median([x[1] for x in runs]))
        chunked.append({"B": B, "sub_batches": -(-nu // B), "mean_completion_ms": round(mean_c, 4),
                        "max_completion_ms": round(max_c, 4),
                        "J_lambda_0.5_ms": round(0.5 * mean_c + 0.5 * max_c, 4)})

    # k sub-batches on k streams (each with its own workspace)
    split = []
    for parts in (1, 2, 4):
        streams = [torch.cuda.Stream(dev) for _ in range(parts)]
        res = []
        for r in range(reps):
            torch.cuda.synchronize(dev)
            a = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for s_ in streams:
                s_.wait_event(a)
            m.score_split(corpus, nu, parts, streams, scale)
            ends = []
            for s_ in streams:
                e = torch.cuda.Event(enable_timing=True)
                e.record(s_)
                ends.append(e)
            torch.cuda.synchronize(dev)
            res.append(max(a.elapsed_time(e) for e in ends))
        split.append({"k": parts, "makespan_ms": round(float(np.median(res)), 4)})

    full = next(c for c in chunked if c["B"] == nu)
    out = {"metric": "score latency vs batch size and micro-batching of the window (Eq. 8)",
           "value": round(nu / full["max_completion_ms"] * 1e3, 1), "unit": "queries/s",
           "n_gpus": 1, "steps": reps, "warmup": 2, "ms_per_step": full["max_completion_ms"],
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": f"{cfg.name}: {cfg.desc}", "n_unique": nu, "k": k,
                      "n_corpus": N, "corpus_layout": "tiled" if tiled else "rows"},
           "latency_curve": curve, "sequential_sub_batches": chunked, "stream_split": split}
    print(json.dumps(out), flush=True)


# weights of the priority function used by the priority modes
PRIO_WEIGHTS = dict(alpha=2.0, gamma=0.75, delta=5.0, eps=0.25)


def priority_bench(args):
    """hs_dedup + hs_priority alone on one workload's requests."""
    import numpy as np
    import torch

    import paper_2607_22578_amd as hs
    import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.make(args.prio_only, seed=args.seed, with_corpus=False)
    phi, s_hat, heavy = synth.scheduler_inputs(w)
    R = w.R
    plan = hs.hs_merge_plan(R, 8, 1, 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    kd = torch.from_numpy(w.keys).to(dev)
    uk = torch.empty(R, dtype=torch.int64, device=dev)
    fi = torch.empty(R, dtype=torch.int32, device=dev)
    ct = torch.empty(R, dtype=torch.int32, device=dev)
    inv = torch.empty(R, dtype=torch.int32, device=dev)
    nu = torch.zeros(1, dtype=torch.int64, device=dev)
    phf = torch.empty(R, dtype=torch.float64, device=dev)
    pi = torch.empty(R, dtype=torch.float64, device=dev)
    order = torch.empty(R, dtype=torch.int32, device=dev)
    ph, sh, hv = (torch.from_numpy(x).to(dev) for x in (phi, s_hat, heavy))
    stream = torch.cuda.Stream(dev)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    d_ms, p_ms = [], []
    for i in range(args.warmup + args.steps):
        evs[0].record(stream)
        hs.hs_dedup(plan, kd, uk, fi, ct, inv, nu, None, ws, stream=stream)
        evs[1].record(stream)
        hs.hs_priority(plan, inv, fi, -1, nu, ph, sh, hv, PRIO_WEIGHTS["alpha"],
                       PRIO_WEIGHTS["gamma"], PRIO_WEIGHTS["delta"], PRIO_WEIGHTS["eps"], phf,
                       pi, order, ws, stream=stream)
        evs[2].record(stream)
        torch.cuda.synchronize(dev)
        if i >= args.warmup:
            d_ms.append(evs[0].elapsed_time(evs[1]))
            p_ms.append(evs[1].elapsed_time(evs[2]))
    n_u = int(nu.item())
    tot = float(np.mean(d_ms)) + float(np.mean(p_ms))
    out = {"metric": "fused-node priorities: requests/s through dedup + priority + order",
           "value": round(R / (tot * 1e-3), 1), "unit": "requests/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(tot, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
           "data": "synthetic",
           "config": {"workload": f"{w.cfg.name}: {w.cfg.desc}", "n_requests": R,
                      "n_unique": n_u, "weights": PRIO_WEIGHTS},
           "dedup_ms": round(float(np.mean(d_ms)), 4),
           "priority_ms": round(float(np.mean(p_ms)), 4)}
    print(json.dumps(out), flush=True)


def oracle_threads(requested: int = 0) -> int:
    """Threads of the CPU baseline: the request, else OMP_NUM_THREADS, else the
    CPUs this process may run on."""
    if requested > 0:
        return requested
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    try:
        return len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        return os.cpu_count() or 1


def host_cpu() -> dict:
    """The host CPU as lscpu reports it (model name, sockets, cores, threads)."""
    info = {"model": "", "logical_cpus": os.cpu_count()}
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            key, _, val = line.partition(":")
            key, val = key.strip(), val.strip()
            if key == "Model name":
                info["model"] = val
            elif key == "Socket(s)":
                info["sockets"] = int(val) if val.isdigit() else val
            elif key == "Core(s) per socket":
                info["cores_per_socket"] = int(val) if val.isdigit() else val
            elif key == "Thread(s) per core":
                info["threads_per_core"] = int(val) if val.isdigit() else val
    except (OSError, ValueError):
        pass
    try:
        info["affinity_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        pass
    return info


# oracle cost per multiply-add and thread (one sequential fp64 sum per score),
# used only to size the bounded CPU-baseline sample to about 20 s
ORACLE_NS_PER_MAC = 1.5
CPU_BASELINE_TARGET_S = 20.0


def cpu_baseline(w, n_u: int, n_sample: int, threads_req: int = 0) -> dict:
    """The oracle on the host: full dedup and representative gather, exact
    scoring + top-k for a seeded sample of distinct queries over the whole
    corpus, extrapolated to all n_u distinct queries."""
    import numpy as np

    import oracle
    threads = oracle_threads(threads_req)
    t0 = time.perf_counter()
    ref = oracle.dedup(w.keys)
    rows = oracle.gather_rows(w.q_req, ref["first_index"])
    t_dedup = time.perf_counter() - t0
    rng = np.random.default_rng(1)
    if n_sample <= 0:
        per_query = w.n_corpus * w.dim * ORACLE_NS_PER_MAC * 1e-9
        n_sample = int(CPU_BASELINE_TARGET_S * threads / max(per_query, 1e-9))
        n_sample = max(threads, n_sample)
    n_sample = min(n_sample, ref["n_unique"])
    sel = np.sort(rng.choice(ref["n_unique"], size=n_sample, replace=False))
    t1 = time.perf_counter()
    oracle.topk_exact(rows, w.corpus, w.k, scale=w.scale, q_rows=sel, threads=threads)
    t_score = time.perf_counter() - t1
    t_full = t_dedup + t_score * ref["n_unique"] / n_sample
    cpu = host_cpu()
    return {"value": round(w.R / t_full, 2), "unit": "queries/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu.get("model", ""), "host": cpu,
            "sample": f"dedup+gather of all {w.R} requests, exact fp64 top-{w.k} of "
                      f"{n_sample}/{ref['n_unique']} distinct queries over all {w.n_corpus} "
                      f"rows ({t_score:.1f} s on {threads} threads), extrapolated to all "
                      "distinct queries",
            "measured_s": round(t_dedup + t_score, 2)}


# The dedup path hs_dedup takes for a window's keys (the rule documented with
# hs_dedup): one workgroup up to 4,096 requests (hash table up to 2,048), then
# direct addressing when max - min < R, else an LSD radix sort with one pass
# per 8 bits of max - min.
def dedup_path(keys) -> str:
    import numpy as np
    R = int(keys.shape[0])
    if R <= 2048:
        return "lds-hash (one workgroup)"
    if R <= 4096:
        return "bitonic (one workgroup)"
    span = int(np.max(keys)) - int(np.min(keys))
    if span < R:
        return f"direct addressing (key range {span + 1})"
    passes = max(1, (span.bit_length() + 7) // 8)
    return f"radix ({passes} passes of 8 bits)"


if __name__ == "__main__":
    main()
