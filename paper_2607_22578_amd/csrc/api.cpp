// Host side of libhsmerge: argument validation, plans, workspace layout and
// kernel launches behind the C ABI declared in include/hs_merge.h.
//
// Every entry point validates all of its arguments before it enqueues
// anything, so a non-OK status means nothing was launched and no output was
// touched.  No entry point allocates device memory.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/hs_merge.h"

namespace hs {
size_t dedup_workspace_bytes(int64_t R);
hipError_t launch_dedup(const int64_t *keys, int64_t R, int64_t *uk, int32_t *fi, int32_t *cnt,
                        int32_t *inv, int64_t *nu, void *ws, hipStream_t st);
hipError_t launch_gather(const void *src, int64_t src_rows, int64_t row_bytes, const void *index,
                         int is64, int64_t n_out, const int64_t *n_out_dev, void *dst,
                         hipStream_t st);
hipError_t launch_deliver(const float *ts, const int32_t *ti, int64_t rows, const int32_t *inv,
                          int64_t R, int k, float *os, int32_t *oi, hipStream_t st);
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void **ptr);
size_t score_workspace_bytes(int64_t cap, int64_t N, int64_t d, int k, int corpus_dtype);
hipError_t launch_score_partial(const void *q, const void *corpus, const float *scale, int64_t N,
                                int64_t d, int k, int64_t n_unique, const int64_t *nu_dev,
                                int64_t cap, int corpus_dtype, bool tiled, void *part,
                                hipStream_t st);
size_t mfma_tiled_bytes(int64_t N, int64_t d, bool fp8);
hipError_t launch_tile_corpus(const void *corpus, int64_t N, int64_t d, bool fp8, void *tiled,
                              hipStream_t st);
hipError_t launch_topk_merge(const void *part, int64_t n_unique, const int64_t *nu_dev,
                             int64_t cap, int64_t N, int k, int corpus_dtype, float *out_s,
                             int32_t *out_i, hipStream_t st);
struct CacheView;
size_t cache_layout(int64_t C, int k, void *base, CacheView *v);
hipError_t launch_cache_reset(void *cache, int64_t C, int k, hipStream_t st);
hipError_t launch_cache_lookup(void *cache, int64_t C, int k, const int64_t *uk,
                               const int32_t *fi, int64_t n_unique, const int64_t *nu_dev,
                               int64_t cap, float *out_s, int32_t *out_i, int32_t *miss_pos,
                               int32_t *miss_first, int64_t *n_miss, hipStream_t st);
hipError_t launch_cache_insert(void *cache, int64_t C, int k, const int64_t *uk, int64_t n_unique,
                               const int64_t *nu_dev, int64_t cap, const int32_t *miss_pos,
                               const float *top_s, const int32_t *top_i, hipStream_t st);
hipError_t launch_signature(const uint32_t *op_type, const uint8_t *params,
                            const int64_t *param_off, int64_t param_bytes, const uint8_t *text,
                            const int64_t *text_off, int64_t text_bytes, const int32_t *pred_off,
                            const int32_t *pred_idx, int64_t pred_count, int64_t first,
                            int64_t count, int normalize, uint8_t *digest, int64_t *keys,
                            hipStream_t st);
size_t priority_workspace_bytes(int64_t cap);
hipError_t launch_priority(const int32_t *inverse, const int32_t *first_index, int64_t R,
                           int64_t n_unique, const int64_t *nu_dev, int64_t cap,
                           const float *phi, const float *s_hat, const uint8_t *heavy,
                           double alpha, double gamma, double delta, double eps, double *phi_out,
                           double *pi_out, int32_t *order, void *ws, hipStream_t st);
}  // namespace hs

struct hs_plan {
  hs_merge_desc d;      // (d.workflow_offsets is not kept: see offsets)
  std::vector<int64_t> offsets;   // workflow CSR [W + 1]
  int64_t cap;          // max distinct keys
  size_t ws_dedup;      // bytes used by hs_dedup (offset 0)
  size_t ws_score;      // bytes used by the score phases (offset 0)
  size_t ws_prio;       // bytes used by hs_priority (offset 0)
  size_t ws_total;
};

static thread_local char g_err[512];

static hs_status fail(hs_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

static hs_status ok() {
  g_err[0] = 0;
  return HS_OK;
}

static bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

static hs_status device_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ok();
  return fail(HS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

extern "C" {

int32_t hs_abi_version(void) { return HS_ABI_VERSION; }

const char *hs_last_error(void) { return g_err; }

const char *hs_status_string(hs_status s) {
  switch (s) {
    case HS_OK: return "HS_OK";
    case HS_ERR_INVALID_ARG: return "HS_ERR_INVALID_ARG";
    case HS_ERR_UNSUPPORTED: return "HS_ERR_UNSUPPORTED";
    case HS_ERR_WORKSPACE: return "HS_ERR_WORKSPACE";
    case HS_ERR_ALIGNMENT: return "HS_ERR_ALIGNMENT";
    case HS_ERR_DEVICE: return "HS_ERR_DEVICE";
  }
  return "HS_ERR_UNKNOWN";
}

hs_status hs_merge_plan(const hs_merge_desc *desc, hs_plan **plan, size_t *workspace_bytes) {
  if (!desc || !plan || !workspace_bytes)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: null argument");
  const hs_merge_desc &d = *desc;
  if ((d.flags & ~HS_FLAG_TILED_CORPUS) != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: unknown flags 0x%x", d.flags);
  // (2^30 keeps every request index and tile offset of the kernels' int32
  // arithmetic far from overflow)
  if (d.n_requests < 0 || d.n_requests > ((int64_t)1 << 30))
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: n_requests %lld out of [0, 2^30]",
                (long long)d.n_requests);
  if (d.n_corpus < 0 || d.n_corpus > INT32_MAX)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: n_corpus %lld out of [0, 2^31-1]",
                (long long)d.n_corpus);
  if (d.dim < 1 || d.dim > 16384)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: dim %lld out of [1, 16384]",
                (long long)d.dim);
  if (d.k < 1 || d.k > 1024)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: k %d out of [1, 1024]", d.k);
  if (d.max_unique < 0 || d.max_unique > d.n_requests)
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: max_unique %lld out of [0, n_requests]",
                (long long)d.max_unique);
  const bool qf32 = d.query_dtype == HS_F32, qbf16 = d.query_dtype == HS_BF16;
  if (!qf32 && !qbf16)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: query_dtype %d unsupported", d.query_dtype);
  if (qf32 && d.corpus_dtype != HS_F32)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: F32 queries need an F32 corpus");
  if (qbf16 && d.corpus_dtype != HS_BF16 && d.corpus_dtype != HS_FP8_E4M3)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: BF16 queries need a BF16 or FP8 corpus");
  if (qf32 && d.dim % 4 != 0)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: F32 needs dim %% 4 == 0");
  if (qbf16 && d.dim % 8 != 0)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: BF16 needs dim %% 8 == 0");
  if (d.corpus_dtype == HS_FP8_E4M3 && d.dim % 16 != 0)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: FP8 corpus needs dim %% 16 == 0");
  if ((d.flags & HS_FLAG_TILED_CORPUS) && d.corpus_dtype == HS_F32)
    return fail(HS_ERR_UNSUPPORTED, "hs_merge_plan: the tiled layout is for BF16/FP8 corpora");
  if (d.n_workflows < 1 || d.n_workflows > ((int64_t)1 << 30))
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: n_workflows %lld out of [1, 2^30]",
                (long long)d.n_workflows);
  const int64_t W = d.n_workflows;
  if (d.workflow_offsets) {
    const int64_t *o = d.workflow_offsets;
    if (o[0] != 0 || o[W] != d.n_requests)
      return fail(HS_ERR_INVALID_ARG,
                  "hs_merge_plan: workflow_offsets must start at 0 and end at n_requests "
                  "(got %lld and %lld)", (long long)o[0], (long long)o[W]);
    for (int64_t w = 0; w < W; ++w)
      if (o[w + 1] < o[w])
        return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: workflow_offsets decrease at %lld",
                    (long long)w);
  } else if (d.n_requests % W != 0) {
    return fail(HS_ERR_INVALID_ARG,
                "hs_merge_plan: %lld workflows do not divide %lld requests (pass "
                "workflow_offsets)", (long long)W, (long long)d.n_requests);
  }
  hs_plan *p = new (std::nothrow) hs_plan;
  if (!p) return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: out of host memory");
  try {
    p->offsets.resize((size_t)W + 1);
  } catch (...) {
    delete p;
    return fail(HS_ERR_INVALID_ARG, "hs_merge_plan: out of host memory");
  }
  for (int64_t w = 0; w <= W; ++w)
    p->offsets[(size_t)w] = d.workflow_offsets ? d.workflow_offsets[w] : w * (d.n_requests / W);
  p->d = d;
  p->d.workflow_offsets = nullptr;
  p->cap = d.max_unique > 0 ? d.max_unique : d.n_requests;
  p->ws_dedup = hs::dedup_workspace_bytes(d.n_requests);
  p->ws_score = hs::score_workspace_bytes(p->cap, d.n_corpus, d.dim, d.k, d.corpus_dtype);
  p->ws_prio = hs::priority_workspace_bytes(p->cap);
  p->ws_total = p->ws_dedup > p->ws_score ? p->ws_dedup : p->ws_score;
  if (p->ws_prio > p->ws_total) p->ws_total = p->ws_prio;
  *plan = p;
  *workspace_bytes = p->ws_total;
  return ok();
}

void hs_plan_destroy(hs_plan *plan) { delete plan; }

hs_status hs_workflow_rows(const hs_plan *plan, int64_t w, int64_t *first, int64_t *count) {
  if (!plan || !first || !count) return fail(HS_ERR_INVALID_ARG, "hs_workflow_rows: null argument");
  if (w < 0 || w >= plan->d.n_workflows)
    return fail(HS_ERR_INVALID_ARG, "hs_workflow_rows: workflow %lld out of [0, %lld)",
                (long long)w, (long long)plan->d.n_workflows);
  *first = plan->offsets[(size_t)w];
  *count = plan->offsets[(size_t)w + 1] - plan->offsets[(size_t)w];
  return ok();
}

hs_status hs_dedup(const hs_plan *plan, const int64_t *keys, int64_t *unique_keys,
                   int32_t *first_index, int32_t *counts, int32_t *inverse,
                   int64_t *n_unique_dev, int64_t *n_unique_host, void *ws, size_t ws_bytes,
                   void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_dedup: null plan");
  const int64_t R = plan->d.n_requests;
  if (!n_unique_dev) return fail(HS_ERR_INVALID_ARG, "hs_dedup: null n_unique_dev");
  if (R > 0 && (!keys || !unique_keys || !first_index || !inverse))
    return fail(HS_ERR_INVALID_ARG, "hs_dedup: null array argument");
  if (!aligned(keys, 8) || !aligned(unique_keys, 8) || !aligned(n_unique_dev, 8) ||
      !aligned(first_index, 4) || !aligned(inverse, 4) || !aligned(counts, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_dedup: misaligned pointer");
  if (plan->ws_dedup > 0 && (!ws || ws_bytes < plan->ws_dedup))
    return fail(HS_ERR_WORKSPACE, "hs_dedup: workspace %zu bytes, need %zu", ws_bytes,
                plan->ws_dedup);
  if (plan->ws_dedup > 0 && !aligned(ws, 256))
    return fail(HS_ERR_ALIGNMENT, "hs_dedup: workspace must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  {
    hipError_t e = hs::launch_dedup(keys, R, unique_keys, first_index, counts, inverse,
                                    n_unique_dev, ws, st);
    if (e != hipSuccess) return device_status(e, "hs_dedup launch");
  }
  if (n_unique_host) {
    hipError_t e = hipMemcpyAsync(n_unique_host, n_unique_dev, sizeof(int64_t),
                                  hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return device_status(e, "hs_dedup readback");
  }
  return ok();
}

static hs_status check_nu(const hs_plan *plan, int64_t n_unique, const int64_t *n_unique_dev,
                          const char *who) {
  if (n_unique == -1) {
    if (!n_unique_dev) return fail(HS_ERR_INVALID_ARG, "%s: n_unique = -1 needs n_unique_dev", who);
    if (!aligned(n_unique_dev, 8)) return fail(HS_ERR_ALIGNMENT, "%s: misaligned n_unique_dev", who);
  } else if (n_unique < 0 || n_unique > plan->cap) {
    return fail(HS_ERR_INVALID_ARG, "%s: n_unique %lld out of [0, %lld]", who,
                (long long)n_unique, (long long)plan->cap);
  }
  return HS_OK;
}

static hs_status check_score_ws(const hs_plan *plan, void *ws, size_t ws_bytes, const char *who) {
  if (plan->ws_score > 0 && (!ws || ws_bytes < plan->ws_score))
    return fail(HS_ERR_WORKSPACE, "%s: workspace %zu bytes, need %zu", who, ws_bytes,
                plan->ws_score);
  if (plan->ws_score > 0 && !aligned(ws, 256))
    return fail(HS_ERR_ALIGNMENT, "%s: workspace must be 256-byte aligned", who);
  return HS_OK;
}

static hs_status check_partial(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                               const int64_t *n_unique_dev, const void *corpus,
                               const float *row_scale, void *ws, size_t ws_bytes,
                               const char *who) {
  hs_status s = check_nu(plan, n_unique, n_unique_dev, who);
  if (s != HS_OK) return s;
  const hs_merge_desc &d = plan->d;
  if (!q_unique && n_unique != 0) return fail(HS_ERR_INVALID_ARG, "%s: null q_unique", who);
  if (!corpus && d.n_corpus > 0) return fail(HS_ERR_INVALID_ARG, "%s: null corpus", who);
  if (d.corpus_dtype == HS_FP8_E4M3 && d.n_corpus > 0 && !row_scale)
    return fail(HS_ERR_INVALID_ARG, "%s: FP8 corpus needs row_scale", who);
  if (!aligned(q_unique, 16) || !aligned(corpus, 16) || !aligned(row_scale, 4))
    return fail(HS_ERR_ALIGNMENT, "%s: q_unique/corpus must be 16-byte aligned", who);
  return check_score_ws(plan, ws, ws_bytes, who);
}

hs_status hs_score_partial(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                           const int64_t *n_unique_dev, const void *corpus,
                           const float *row_scale, void *ws, size_t ws_bytes, void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_score_partial: null plan");
  hs_status s = check_partial(plan, q_unique, n_unique, n_unique_dev, corpus, row_scale, ws,
                              ws_bytes, "hs_score_partial");
  if (s != HS_OK) return s;
  const hs_merge_desc &d = plan->d;
  hipError_t e = hs::launch_score_partial(q_unique, corpus, row_scale, d.n_corpus, d.dim, d.k,
                                          n_unique, n_unique_dev, plan->cap, d.corpus_dtype,
                                          (d.flags & HS_FLAG_TILED_CORPUS) != 0, ws,
                                          (hipStream_t)stream);
  return device_status(e, "hs_score_partial launch");
}

hs_status hs_topk_merge(const hs_plan *plan, int64_t n_unique, const int64_t *n_unique_dev,
                        float *topk_score, int32_t *topk_index, void *ws, size_t ws_bytes,
                        void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_topk_merge: null plan");
  hs_status s = check_nu(plan, n_unique, n_unique_dev, "hs_topk_merge");
  if (s != HS_OK) return s;
  if ((!topk_score || !topk_index) && n_unique != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_topk_merge: null output");
  if (!aligned(topk_score, 4) || !aligned(topk_index, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_topk_merge: misaligned output");
  s = check_score_ws(plan, ws, ws_bytes, "hs_topk_merge");
  if (s != HS_OK) return s;
  const hs_merge_desc &d = plan->d;
  hipError_t e = hs::launch_topk_merge(ws, n_unique, n_unique_dev, plan->cap, d.n_corpus, d.k,
                                       d.corpus_dtype, topk_score, topk_index,
                                       (hipStream_t)stream);
  return device_status(e, "hs_topk_merge launch");
}

hs_status hs_score_topk(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                        const int64_t *n_unique_dev, const void *corpus, const float *row_scale,
                        float *topk_score, int32_t *topk_index, void *ws, size_t ws_bytes,
                        void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_score_topk: null plan");
  hs_status s = check_partial(plan, q_unique, n_unique, n_unique_dev, corpus, row_scale, ws,
                              ws_bytes, "hs_score_topk");
  if (s != HS_OK) return s;
  if ((!topk_score || !topk_index) && n_unique != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_score_topk: null output");
  if (!aligned(topk_score, 4) || !aligned(topk_index, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_score_topk: misaligned output");
  s = hs_score_partial(plan, q_unique, n_unique, n_unique_dev, corpus, row_scale, ws, ws_bytes,
                       stream);
  if (s != HS_OK) return s;
  return hs_topk_merge(plan, n_unique, n_unique_dev, topk_score, topk_index, ws, ws_bytes,
                       stream);
}

hs_status hs_score_topk_noalloc(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                                const int64_t *n_unique_dev, const void *corpus,
                                const float *row_scale, float *topk_score, int32_t *topk_index,
                                void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_score_topk_noalloc: null plan");
  const size_t cap_bytes = hs::noalloc_scratch_bytes();
  if (plan->ws_score > cap_bytes)
    return fail(HS_ERR_WORKSPACE,
                "hs_score_topk_noalloc: this plan's score step needs %zu bytes of scratch, more "
                "than the %zu bytes the library holds per GPU (use hs_score_topk with a "
                "workspace)", plan->ws_score, cap_bytes);
  // validation of everything but the workspace, before any device call
  hs_status s = check_nu(plan, n_unique, n_unique_dev, "hs_score_topk_noalloc");
  if (s != HS_OK) return s;
  const hs_merge_desc &d = plan->d;
  if (!q_unique && n_unique != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_score_topk_noalloc: null q_unique");
  if (!corpus && d.n_corpus > 0)
    return fail(HS_ERR_INVALID_ARG, "hs_score_topk_noalloc: null corpus");
  if (d.corpus_dtype == HS_FP8_E4M3 && d.n_corpus > 0 && !row_scale)
    return fail(HS_ERR_INVALID_ARG, "hs_score_topk_noalloc: FP8 corpus needs row_scale");
  if (!aligned(q_unique, 16) || !aligned(corpus, 16) || !aligned(row_scale, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_score_topk_noalloc: q_unique/corpus must be 16-byte aligned");
  if ((!topk_score || !topk_index) && n_unique != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_score_topk_noalloc: null output");
  if (!aligned(topk_score, 4) || !aligned(topk_index, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_score_topk_noalloc: misaligned output");
  void *ws = nullptr;
  hipError_t e = hs::noalloc_scratch(&ws);
  if (e != hipSuccess) return device_status(e, "hs_score_topk_noalloc scratch");
  hipStream_t st = (hipStream_t)stream;
  e = hs::launch_score_partial(q_unique, corpus, row_scale, d.n_corpus, d.dim, d.k, n_unique,
                               n_unique_dev, plan->cap, d.corpus_dtype,
                               (d.flags & HS_FLAG_TILED_CORPUS) != 0, ws, st);
  if (e != hipSuccess) return device_status(e, "hs_score_topk_noalloc launch");
  e = hs::launch_topk_merge(ws, n_unique, n_unique_dev, plan->cap, d.n_corpus, d.k,
                            d.corpus_dtype, topk_score, topk_index, st);
  return device_status(e, "hs_score_topk_noalloc launch");
}

hs_status hs_corpus_tiled_bytes(const hs_plan *plan, size_t *bytes) {
  if (!plan || !bytes) return fail(HS_ERR_INVALID_ARG, "hs_corpus_tiled_bytes: null argument");
  const hs_merge_desc &d = plan->d;
  if (d.corpus_dtype == HS_F32)
    return fail(HS_ERR_UNSUPPORTED, "hs_corpus_tiled_bytes: the tiled layout is for BF16/FP8 "
                "corpora");
  *bytes = hs::mfma_tiled_bytes(d.n_corpus, d.dim, d.corpus_dtype == HS_FP8_E4M3);
  return HS_OK;
}

hs_status hs_tile_corpus(const hs_plan *plan, const void *corpus, void *tiled,
                         size_t tiled_bytes, void *stream) {
  size_t need = 0;
  hs_status s = hs_corpus_tiled_bytes(plan, &need);
  if (s != HS_OK) return s;
  const hs_merge_desc &d = plan->d;
  if (!corpus && d.n_corpus > 0) return fail(HS_ERR_INVALID_ARG, "hs_tile_corpus: null corpus");
  if (!tiled && need > 0) return fail(HS_ERR_INVALID_ARG, "hs_tile_corpus: null tiled buffer");
  if (tiled_bytes < need)
    return fail(HS_ERR_INVALID_ARG, "hs_tile_corpus: tiled buffer of %zu bytes, %zu needed",
                tiled_bytes, need);
  if (!aligned(corpus, 16) || !aligned(tiled, 16))
    return fail(HS_ERR_ALIGNMENT, "hs_tile_corpus: corpus/tiled must be 16-byte aligned");
  if (corpus && tiled && need > 0) {
    // the source rows and the tiled buffer must not overlap
    const uintptr_t c0 = (uintptr_t)corpus, t0 = (uintptr_t)tiled;
    const size_t cb = (size_t)d.n_corpus * (size_t)d.dim *
                      (d.corpus_dtype == HS_FP8_E4M3 ? 1u : 2u);
    if (c0 < t0 + need && t0 < c0 + cb)
      return fail(HS_ERR_INVALID_ARG, "hs_tile_corpus: corpus and tiled buffer overlap");
  }
  hipError_t e = hs::launch_tile_corpus(corpus, d.n_corpus, d.dim,
                                        d.corpus_dtype == HS_FP8_E4M3, tiled,
                                        (hipStream_t)stream);
  return device_status(e, "hs_tile_corpus launch");
}

hs_status hs_scatter(const void *src, int64_t src_rows, int64_t row_bytes, const void *index,
                     int32_t index_is_i64, int64_t n_out, const int64_t *n_out_dev, void *dst,
                     void *stream) {
  if (src_rows < 0 || n_out < 0)
    return fail(HS_ERR_INVALID_ARG, "hs_scatter: negative size");
  if (row_bytes <= 0 || row_bytes % 4 != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_scatter: row_bytes %lld must be a positive multiple of 4",
                (long long)row_bytes);
  if (index_is_i64 != 0 && index_is_i64 != 1)
    return fail(HS_ERR_INVALID_ARG, "hs_scatter: index_is_i64 must be 0 or 1");
  if (n_out > 0 && src_rows > 0 && (!src || !index || !dst))
    return fail(HS_ERR_INVALID_ARG, "hs_scatter: null argument");
  if (!aligned(src, 4) || !aligned(dst, 4) || !aligned(index, index_is_i64 ? 8 : 4) ||
      !aligned(n_out_dev, 8))
    return fail(HS_ERR_ALIGNMENT, "hs_scatter: misaligned pointer");
  if (n_out == 0 || src_rows == 0) return ok();
  hipError_t e = hs::launch_gather(src, src_rows, row_bytes, index, index_is_i64, n_out,
                                   n_out_dev, dst, (hipStream_t)stream);
  return device_status(e, "hs_scatter launch");
}

hs_status hs_deliver(const hs_plan *plan, const float *topk_score, const int32_t *topk_index,
                     int64_t topk_rows, const int32_t *inverse, float *out_score,
                     int32_t *out_index, void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_deliver: null plan");
  if (topk_rows < 0) return fail(HS_ERR_INVALID_ARG, "hs_deliver: negative topk_rows");
  const int64_t R = plan->d.n_requests;
  if (R == 0 || topk_rows == 0) return ok();
  if (!topk_score || !topk_index || !inverse || !out_score || !out_index)
    return fail(HS_ERR_INVALID_ARG, "hs_deliver: null argument");
  if (!aligned(topk_score, 4) || !aligned(topk_index, 4) || !aligned(inverse, 4) ||
      !aligned(out_score, 4) || !aligned(out_index, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_deliver: misaligned pointer");
  hipError_t e = hs::launch_deliver(topk_score, topk_index, topk_rows, inverse, R, plan->d.k,
                                    out_score, out_index, (hipStream_t)stream);
  return device_status(e, "hs_deliver launch");
}

// ---------------------------------------------------------------- result store

static hs_status check_cache(const hs_plan *plan, const void *cache, size_t cache_bytes,
                             int64_t capacity, const char *who) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "%s: null plan", who);
  if (capacity < 1 || capacity > ((int64_t)1 << 30) || (capacity & (capacity - 1)) != 0)
    return fail(HS_ERR_INVALID_ARG, "%s: capacity %lld must be a power of two in [1, 2^30]", who,
                (long long)capacity);
  if (!cache) return fail(HS_ERR_INVALID_ARG, "%s: null cache", who);
  if (!aligned(cache, 256)) return fail(HS_ERR_ALIGNMENT, "%s: cache not 256-byte aligned", who);
  const size_t need = hs::cache_layout(capacity, plan->d.k, nullptr, nullptr);
  if (cache_bytes < need)
    return fail(HS_ERR_WORKSPACE, "%s: cache has %zu bytes, needs %zu", who, cache_bytes, need);
  return ok();
}

hs_status hs_cache_bytes(const hs_plan *plan, int64_t capacity, size_t *bytes) {
  if (!plan || !bytes) return fail(HS_ERR_INVALID_ARG, "hs_cache_bytes: null argument");
  if (capacity < 1 || capacity > ((int64_t)1 << 30) || (capacity & (capacity - 1)) != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_cache_bytes: capacity %lld must be a power of two in "
                "[1, 2^30]", (long long)capacity);
  *bytes = hs::cache_layout(capacity, plan->d.k, nullptr, nullptr);
  return ok();
}

hs_status hs_cache_reset(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                         void *stream) {
  hs_status s = check_cache(plan, cache, cache_bytes, capacity, "hs_cache_reset");
  if (s != HS_OK) return s;
  hipError_t e = hs::launch_cache_reset(cache, capacity, plan->d.k, (hipStream_t)stream);
  return device_status(e, "hs_cache_reset launch");
}

hs_status hs_cache_lookup(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                          const int64_t *unique_keys, const int32_t *first_index,
                          int64_t n_unique, const int64_t *n_unique_dev, float *topk_score,
                          int32_t *topk_index, int32_t *miss_pos, int32_t *miss_first,
                          int64_t *n_miss_dev, void *stream) {
  hs_status s = check_cache(plan, cache, cache_bytes, capacity, "hs_cache_lookup");
  if (s != HS_OK) return s;
  s = check_nu(plan, n_unique, n_unique_dev, "hs_cache_lookup");
  if (s != HS_OK) return s;
  if (!unique_keys || !first_index || !topk_score || !topk_index || !miss_pos || !miss_first ||
      !n_miss_dev)
    return fail(HS_ERR_INVALID_ARG, "hs_cache_lookup: null argument");
  if (!aligned(unique_keys, 8) || !aligned(n_miss_dev, 8) || !aligned(first_index, 4) ||
      !aligned(topk_score, 4) || !aligned(topk_index, 4) || !aligned(miss_pos, 4) ||
      !aligned(miss_first, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_cache_lookup: misaligned pointer");
  hipError_t e = hs::launch_cache_lookup(cache, capacity, plan->d.k, unique_keys, first_index,
                                         n_unique, n_unique_dev, plan->cap, topk_score,
                                         topk_index, miss_pos, miss_first, n_miss_dev,
                                         (hipStream_t)stream);
  return device_status(e, "hs_cache_lookup launch");
}

hs_status hs_cache_insert(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                          const int64_t *unique_keys, const int32_t *miss_pos, int64_t n_unique,
                          const int64_t *n_unique_dev, const float *topk_score,
                          const int32_t *topk_index, void *stream) {
  hs_status s = check_cache(plan, cache, cache_bytes, capacity, "hs_cache_insert");
  if (s != HS_OK) return s;
  s = check_nu(plan, n_unique, n_unique_dev, "hs_cache_insert");
  if (s != HS_OK) return s;
  if (!unique_keys || !miss_pos || !topk_score || !topk_index)
    return fail(HS_ERR_INVALID_ARG, "hs_cache_insert: null argument");
  if (!aligned(unique_keys, 8) || !aligned(miss_pos, 4) || !aligned(topk_score, 4) ||
      !aligned(topk_index, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_cache_insert: misaligned pointer");
  hipError_t e = hs::launch_cache_insert(cache, capacity, plan->d.k, unique_keys, n_unique,
                                         n_unique_dev, plan->cap, miss_pos, topk_score,
                                         topk_index, (hipStream_t)stream);
  return device_status(e, "hs_cache_insert launch");
}

// ---------------------------------------------------------------- signatures

hs_status hs_signature(const hs_sig_nodes *nd, int64_t first, int64_t count, int32_t flags,
                       uint8_t *digest, int64_t *keys, void *stream) {
  if (!nd) return fail(HS_ERR_INVALID_ARG, "hs_signature: null node description");
  const int64_t kMaxBuf = ((int64_t)1 << 32) - 16;
  if (nd->n_nodes < 0 || nd->n_nodes > ((int64_t)1 << 27))
    return fail(HS_ERR_INVALID_ARG, "hs_signature: n_nodes %lld out of [0, 2^27]",
                (long long)nd->n_nodes);
  if (first < 0 || count < 0 || first > nd->n_nodes - count)
    return fail(HS_ERR_INVALID_ARG, "hs_signature: range [%lld, +%lld) outside [0, %lld)",
                (long long)first, (long long)count, (long long)nd->n_nodes);
  if ((flags & ~HS_SIG_NORMALIZE_TEXT) != 0)
    return fail(HS_ERR_INVALID_ARG, "hs_signature: unknown flags 0x%x", flags);
  if (nd->param_bytes < 0 || nd->param_bytes > kMaxBuf || nd->text_bytes < 0 ||
      nd->text_bytes > kMaxBuf)
    return fail(HS_ERR_INVALID_ARG, "hs_signature: buffer sizes must be in [0, 2^32 - 16]");
  if (nd->pred_count < 0 || nd->pred_count > INT32_MAX)
    return fail(HS_ERR_INVALID_ARG, "hs_signature: pred_count out of [0, 2^31 - 1]");
  if (count == 0) return ok();
  if (!nd->op_type || !digest)
    return fail(HS_ERR_INVALID_ARG, "hs_signature: null op_type or digest");
  if ((nd->param_off && nd->param_bytes > 0 && !nd->params) ||
      (nd->text_off && nd->text_bytes > 0 && !nd->text) ||
      (nd->pred_off && nd->pred_count > 0 && !nd->pred_idx))
    return fail(HS_ERR_INVALID_ARG, "hs_signature: null data buffer with a non-zero size");
  if (!aligned(digest, 16) || !aligned(keys, 8) || !aligned(nd->op_type, 4) ||
      !aligned(nd->param_off, 8) || !aligned(nd->text_off, 8) || !aligned(nd->pred_off, 4) ||
      !aligned(nd->pred_idx, 4))
    return fail(HS_ERR_ALIGNMENT, "hs_signature: misaligned pointer");
  hipError_t e = hs::launch_signature(
      nd->op_type, nd->params, nd->param_off, nd->params ? nd->param_bytes : 0, nd->text,
      nd->text_off, nd->text ? nd->text_bytes : 0, nd->pred_off, nd->pred_idx,
      nd->pred_idx ? nd->pred_count : 0, first, count, (flags & HS_SIG_NORMALIZE_TEXT) ? 1 : 0,
      digest, keys, (hipStream_t)stream);
  return device_status(e, "hs_signature launch");
}

// ---------------------------------------------------------------- priorities

hs_status hs_priority(const hs_plan *plan, const int32_t *inverse, const int32_t *first_index,
                      int64_t n_unique, const int64_t *n_unique_dev, const float *phi,
                      const float *s_hat, const uint8_t *heavy, double alpha, double gamma,
                      double delta, double eps, double *phi_fused, double *pi, int32_t *order,
                      void *ws, size_t ws_bytes, void *stream) {
  if (!plan) return fail(HS_ERR_INVALID_ARG, "hs_priority: null plan");
  hs_status s = check_nu(plan, n_unique, n_unique_dev, "hs_priority");
  if (s != HS_OK) return s;
  if (!std::isfinite(alpha) || !std::isfinite(gamma) || !std::isfinite(delta) ||
      !std::isfinite(eps) || !(eps > 0.0))
    return fail(HS_ERR_INVALID_ARG, "hs_priority: alpha, gamma, delta must be finite and eps > 0");
  if (n_unique == 0) return ok();
  if (!inverse || !first_index || !phi || !s_hat || !order)
    return fail(HS_ERR_INVALID_ARG, "hs_priority: null argument");
  if (!ws || ws_bytes < plan->ws_prio)
    return fail(HS_ERR_WORKSPACE, "hs_priority: workspace has %zu bytes, needs %zu", ws_bytes,
                plan->ws_prio);
  if (!aligned(ws, 256)) return fail(HS_ERR_ALIGNMENT, "hs_priority: workspace not 256-aligned");
  if (!aligned(inverse, 4) || !aligned(first_index, 4) || !aligned(phi, 4) ||
      !aligned(s_hat, 4) || !aligned(order, 4) || !aligned(phi_fused, 8) || !aligned(pi, 8))
    return fail(HS_ERR_ALIGNMENT, "hs_priority: misaligned pointer");
  hipError_t e = hs::launch_priority(inverse, first_index, plan->d.n_requests, n_unique,
                                     n_unique_dev, plan->cap, phi, s_hat, heavy, alpha, gamma,
                                     delta, eps, phi_fused, pi, order, ws, (hipStream_t)stream);
  return device_status(e, "hs_priority launch");
}

}  // extern "C"
