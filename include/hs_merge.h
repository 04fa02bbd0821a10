/*
 * hs_merge.h -- C ABI of libhsmerge.so: merged retrieval on one MI355X (gfx950).
 *
 * Many concurrent workflows issue embedding-retrieval nodes over one shared
 * chunk corpus.  Following HeraSys (Li et al.), Sec. 3.3 "Pre-Execution
 * Optimization: Semantic Graph Fusion":
 *   - each node carries a semantic signature (Eq. 2); nodes with equal
 *     signatures are computationally equivalent;
 *   - within a time window, a duplicate node is removed, its downstream edges
 *     are redirected to the surviving node, and the survivor's output flows to
 *     every related query (Topological Fusion within Time Window);
 *   - same-type ready nodes execute as one batch (Appendix A, batching
 *     constraint: b <= B_r, only nodes with consistent profile).
 * The library runs that window as device steps on a caller stream:
 *   hs_dedup       group the R request keys (signatures) -> distinct keys,
 *                  survivor per group, group sizes |M(v*)| (Eq. 3), and the
 *                  redirect map request -> group;
 *   hs_scatter     row gather: representative query rows and embedding rows
 *                  of distinct chunk ids;
 *   hs_score_topk  exact inner-product top-k of every distinct query against
 *                  the corpus (retrieval with Top-K among its parameters,
 *                  Eq. 2; top-K vector retrieval of the RAG workloads, Sec. 4.1)
 *                  = hs_score_partial followed by hs_topk_merge;
 *   hs_deliver     every request receives its group's result, each
 *                  workflow's requests in one contiguous row range.
 * Optionally, hs_cache_lookup / hs_cache_insert reuse results across windows
 * (Sec. 3.3 (II)), so that only keys not seen before are scored,
 * hs_signature computes the keys themselves from node descriptions (Eq. 2),
 * and hs_priority ranks the fused nodes for the ready queue (Eq. 3, Eq. 7).
 *
 * Conventions (all entry points):
 *   - Every function returns hs_status.  Arguments are validated on the host
 *     before anything is enqueued; on a non-OK status nothing was enqueued and
 *     no output was written.  hs_last_error() gives a message (thread-local).
 *   - Device pointers are plain addresses in the current HIP device's memory,
 *     owned by the caller; the library never allocates or frees device memory
 *     and keeps no pointer after a call returns.  Temporary device memory comes
 *     from a caller-provided workspace (ws, ws_bytes) sized by hs_merge_plan.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All work is asynchronous on that stream; outputs are valid after the
 *     stream is synchronised.  The only host synchronisation the library ever
 *     performs is the optional n_unique_host readback of hs_dedup.
 *   - Layout: row-major and contiguous (a BF16/FP8 corpus may instead be in
 *     the tiled layout of hs_tile_corpus).  Row data pointers must be 16-byte
 *     aligned; integer arrays must be aligned to their element size.
 *   - Device-side faults (e.g. an out-of-range index inside device data) cannot
 *     be reported synchronously: kernels skip such entries instead of reading
 *     out of bounds, and document what they leave in the output.
 */
#ifndef HS_MERGE_H
#define HS_MERGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HS_ABI_VERSION 3

typedef enum {
    HS_OK = 0,
    HS_ERR_INVALID_ARG = 1,   /* null/negative/inconsistent argument */
    HS_ERR_UNSUPPORTED = 2,   /* dtype / dim / k combination not implemented */
    HS_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required */
    HS_ERR_ALIGNMENT = 4,     /* pointer not aligned as required */
    HS_ERR_DEVICE = 5         /* a HIP call failed (message in hs_last_error) */
} hs_status;

typedef enum {
    HS_F32 = 0,        /* IEEE binary32 */
    HS_BF16 = 1,       /* bfloat16 (upper half of binary32), stored as uint16 */
    HS_FP8_E4M3 = 2    /* OCP fp8 E4M3 ("fn": bias 7, max 448, no inf), uint8 */
} hs_dtype;

/* Shape of one merge window (one call sequence). */
typedef struct {
    int64_t n_requests;   /* R, 0 <= R <= 2^30: retrieval nodes in the window, in
                             arrival order */
    int64_t dim;          /* d: vector width; F32: d % 4 == 0, BF16: d % 8 == 0,
                             FP8 corpus: d % 16 == 0; 1 <= d <= 16384 */
    int64_t n_corpus;     /* N: corpus rows, 0 <= N <= 2^31 - 1 */
    int32_t k;            /* results per node, 1 <= k <= 1024 (k > N pads) */
    int32_t query_dtype;  /* HS_F32 or HS_BF16 */
    int32_t corpus_dtype; /* HS_F32 (with F32 queries), HS_BF16 or HS_FP8_E4M3
                             (with BF16 queries) */
    int32_t flags;        /* 0 or HS_FLAG_TILED_CORPUS (BF16/FP8 corpora only):
                             the corpus argument of the score calls is then
                             the tiled copy made by hs_tile_corpus */
    int64_t max_unique;   /* batch limit B_r of Appendix A (0 = n_requests): the
                             score step handles at most this many distinct
                             queries per call; a window with more distinct keys
                             is scored in several batches (see hs_score_topk) */
    int64_t n_workflows;  /* W >= 1: workflows that issued the window's requests
                             (Sec. 3.3 (I): the fused nodes of several
                             concurrent workflows) */
    const int64_t *workflow_offsets;
                          /* host CSR [W + 1], may be NULL: workflow w issued
                             requests [off[w], off[w+1]) (arrival order is
                             workflow-major), so its results are those rows of
                             the per-request outputs.  off[0] = 0, non-decreasing,
                             off[W] = n_requests.  NULL = uniform: W divides
                             n_requests and every workflow has n_requests / W.
                             Read and copied during hs_merge_plan only. */
} hs_merge_desc;

/* hs_merge_desc.flags: the score calls read the corpus in the tiled layout. */
#define HS_FLAG_TILED_CORPUS 1

typedef struct hs_plan hs_plan;   /* opaque, immutable, thread-safe host object */

/* Validate `desc` and create a plan.  *workspace_bytes receives the size of the
 * device workspace that hs_dedup and hs_score_topk (and its two phases) need
 * for this shape (it also covers hs_priority).  The plan is freed with
 * hs_plan_destroy.  Bad workflow offsets (wrong first or last entry, a
 * decreasing entry, W not dividing R when they are NULL) are rejected with
 * HS_ERR_INVALID_ARG. */
hs_status hs_merge_plan(const hs_merge_desc *desc, hs_plan **plan, size_t *workspace_bytes);

void hs_plan_destroy(hs_plan *plan);

/* Rows of workflow w (0 <= w < W) in the per-request outputs (hs_deliver):
 * [*first, *first + *count).  Host only, no device work (Sec. 3.3 (I): each
 * workflow's merged nodes receive the survivors' outputs). */
hs_status hs_workflow_rows(const hs_plan *plan, int64_t w, int64_t *first, int64_t *count);

/* Step 1 -- signature matching (Sec. 3.3 (I); Appendix B.3, Phase 1: duplicate
 * detection through a global duplication map).
 *   keys          [R] int64 device: signature of request i (arrival order)
 *   unique_keys   [R cap] int64 device out: distinct keys ascending (signed)
 *   first_index   [R cap] int32 device out: earliest request of each group
 *                 (the surviving node v_e)
 *   counts        [R cap] int32 device out, may be NULL: group sizes |M(v*)|
 *   inverse       [R] int32 device out: group of request i (redirected edge)
 *   n_unique_dev  int64 device out: number of groups n_u
 *   n_unique_host int64 host out, may be NULL: if given, the call waits for
 *                 the stream once and stores n_u there
 * Entries [n_u, R) of the per-group outputs are left unspecified.  R = 0 sets
 * n_u = 0.  Bit-exact and deterministic.  n_unique_dev (and n_unique_host)
 * always hold the full count, even when it exceeds max_unique.
 * Method (for any int64 keys; the outputs do not depend on it): one workgroup
 * for R <= 4,096 (an LDS hash table up to 2,048 requests, else a bitonic sort);
 * above, the key range is found on the device and the keys are numbered by
 * direct addressing when max - min < R, else sorted by an LSD radix sort with
 * one pass per 8 bits of max - min. */
hs_status hs_dedup(const hs_plan *plan, const int64_t *keys, int64_t *unique_keys,
                   int32_t *first_index, int32_t *counts, int32_t *inverse,
                   int64_t *n_unique_dev, int64_t *n_unique_host,
                   void *ws, size_t ws_bytes, void *stream);

/* Steps 3+4 -- one exact top-k retrieval per distinct node over the corpus.
 *   q_unique      [n_u x d] device, query_dtype: representative query rows
 *   n_unique      host count n_u, or -1 to read it from n_unique_dev on the
 *                 device (the launch then covers max_unique rows)
 *   n_unique_dev  int64 device, used when n_unique == -1 (else may be NULL)
 *   corpus        [N x d] device, corpus_dtype; with HS_FLAG_TILED_CORPUS the
 *                 tiled copy of it (hs_tile_corpus), same scores and results
 *   row_scale     [N] fp32 device: per-row dequantisation scale, FP8 only
 *                 (score = row_scale[c] * <q, decode(C[c])>), else NULL
 *   topk_score    [n_u x k] fp32 device out: best scores, descending
 *   topk_index    [n_u x k] int32 device out: corpus rows; equal scores are
 *                 ordered by ascending row; slots beyond N are (-inf, -1)
 * Scores accumulate in fp32 from exact bf16/fp8 products (fp32 products for
 * F32 inputs).  Identical corpus rows get bit-identical scores.
 * One call is one batch of at most max_unique distinct queries (B_r): with
 * n_unique = -1 it scores the first min(n_u, max_unique) rows of q_unique.  A
 * window with more distinct keys than max_unique (n_unique_dev tells) is
 * scored in further calls on the following rows, with host counts and
 * pointers advanced by the batch (topk_score/index then need room for n_u
 * rows). */
hs_status hs_score_topk(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                        const int64_t *n_unique_dev, const void *corpus,
                        const float *row_scale, float *topk_score, int32_t *topk_index,
                        void *ws, size_t ws_bytes, void *stream);

/* hs_score_topk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation and results, with the scratch memory taken from an
 * array the library holds on each GPU (64 MiB per GPU, allocated with the
 * library's code object and kept until the process ends) instead of a
 * workspace argument.  No hipMalloc, hipFree or other allocation happens in
 * the call.  A plan whose score workspace (what hs_merge_plan reports for the
 * score step) exceeds 64 MiB is rejected with HS_ERR_WORKSPACE before
 * anything is enqueued; the 1M-row window (2,048 requests, d = 768, k = 10)
 * needs about 62 MiB.  Every call on one GPU uses that GPU's one array, which
 * keeps the previous call's contents (each call writes everything it reads
 * before reading it): calls that overlap in time on one GPU -- on different
 * streams, or from host threads without ordering -- race and give wrong
 * results; order them on one stream.  Arguments as for hs_score_topk. */
hs_status hs_score_topk_noalloc(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                                const int64_t *n_unique_dev, const void *corpus,
                                const float *row_scale, float *topk_score, int32_t *topk_index,
                                void *stream);

/* Storage layout of a BF16 or FP8 corpus for the score calls (not a step of the
 * method: the corpus of the retrieval nodes, Sec. 3.3 (I) / Sec. 4.1, stored in
 * the order the score kernel copies it, so that each copy reads consecutive
 * bytes; scores and results are the same as from the row-major corpus).
 * Blocks of 384 rows x 64 columns, block (t, s) at byte (t * ceil(d / 64) + s)
 * * 384 * 64 * esz (esz = 2 for BF16, 1 for FP8), each block row-major with the
 * 16-byte pieces of row r permuted within the row (piece p in slot p XOR a
 * function of r mod 16); rows past N and columns past d hold zeros.  A corpus
 * is tiled once and scored in any number of windows.
 * hs_corpus_tiled_bytes: *bytes = size of the tiled copy for the plan's
 *   corpus shape (ceil(N / 384) * 384 * ceil(d / 64) * 64 * esz);
 *   HS_ERR_UNSUPPORTED for an F32 corpus.
 * hs_tile_corpus: writes the tiled copy of `corpus` ([N x d] row-major device,
 *   corpus_dtype) to `tiled` (device, tiled_bytes >= hs_corpus_tiled_bytes,
 *   not overlapping `corpus`; both 16-byte aligned), asynchronously on
 *   `stream`.  The plan's flags need not include HS_FLAG_TILED_CORPUS; plans
 *   that score the tiled copy must. */
hs_status hs_corpus_tiled_bytes(const hs_plan *plan, size_t *bytes);
hs_status hs_tile_corpus(const hs_plan *plan, const void *corpus, void *tiled,
                         size_t tiled_bytes, void *stream);

/* Phase 1 of hs_score_topk: scores every distinct query against the corpus in
 * one persistent kernel, each workgroup keeping the k best (score, row) pairs
 * of its corpus slice per query; the per-slice lists go to the workspace
 * (for BF16/FP8 corpora, together with a per-query lower bound of the k-th
 * best score, which phase 2 uses to drop list entries early; the workspace
 * also holds a copy of the distinct queries in the kernel's tiled order,
 * written by the call itself, so q_unique is only read).
 * Arguments as for hs_score_topk. */
hs_status hs_score_partial(const hs_plan *plan, const void *q_unique, int64_t n_unique,
                           const int64_t *n_unique_dev, const void *corpus,
                           const float *row_scale, void *ws, size_t ws_bytes, void *stream);

/* Phase 2 of hs_score_topk: merges the per-slice lists left in the workspace
 * by hs_score_partial (same plan, same n_unique arguments, same workspace)
 * into the final sorted top-k per distinct query. */
hs_status hs_topk_merge(const hs_plan *plan, int64_t n_unique, const int64_t *n_unique_dev,
                        float *topk_score, int32_t *topk_index,
                        void *ws, size_t ws_bytes, void *stream);

/* Steps 2 and 2' -- row gather dst[i] = src[index[i]], i < n_rows.
 * The race-free form of handing one row to many consumers (Sec. 3.3 (I): one
 * execution instance per merged set, its output flowing to all related
 * queries):
 *   representative rows: src = request queries,  index = first_index
 *   embedding rows:      src = embedding table,  index = unique_keys (int64)
 *   one delivered array: src = topk_score or topk_index, index = inverse
 *                        (hs_deliver does both arrays in one launch)
 *   src        [src_rows x row_bytes] device
 *   row_bytes  > 0 and a multiple of 4 (16-byte rows use 128-bit accesses)
 *   index      [n_out] int32 (index_is_i64 = 0) or int64 (= 1) device
 *   n_out      host row count (upper bound when n_out_dev is given)
 *   n_out_dev  int64 device, may be NULL: actual row count (<= n_out), e.g.
 *              n_unique_dev from hs_dedup
 *   dst        [n_out x row_bytes] device out
 * Rows whose index falls outside [0, src_rows) are left unwritten. */
hs_status hs_scatter(const void *src, int64_t src_rows, int64_t row_bytes,
                     const void *index, int32_t index_is_i64, int64_t n_out,
                     const int64_t *n_out_dev, void *dst, void *stream);

/* Step 5 -- delivery (Sec. 3.3 (I): the survivor's output flows to the
 * downstream nodes of every merged query): for every request i < R,
 *   out_score[i] = topk_score[inverse[i]], out_index[i] = topk_index[inverse[i]]
 * (k entries each, the plan's R and k), in one launch.
 *   topk_score/index [topk_rows x k] device: results of the distinct queries
 *   topk_rows       rows held by topk_score/index (>= 0); a request whose group
 *                   is outside [0, topk_rows) is left unwritten
 *   inverse         [R] int32 device: hs_dedup's request -> group map
 *   out_score/index [R x k] device out: per-request results; workflow w's
 *                   requests are rows hs_workflow_rows(plan, w)
 * Bit-exact copies. */
hs_status hs_deliver(const hs_plan *plan, const float *topk_score, const int32_t *topk_index,
                     int64_t topk_rows, const int32_t *inverse, float *out_score,
                     int32_t *out_index, void *stream);

/* Cross-window reuse (Sec. 3.3 (II), asynchronous cache reuse): a node whose
 * signature matches a node completed in an earlier window takes that node's
 * result instead of being executed again.  The store lives in one caller-owned
 * device buffer and holds at most `capacity` top-k rows of the plan's k:
 *   layout   keys [C] int64 | valid [C] int32 | claim [C] int32 |
 *            score [C x k] fp32 | index [C x k] int32, each array starting on a
 *            256-byte boundary (C = capacity, a power of two in [1, 2^30]);
 *   mapping  direct-mapped, slot(key) = top log2(C) bits of
 *            key * 0x9E3779B97F4A7C15 (mod 2^64), one entry per slot; a hit
 *            needs a valid slot holding the same key;
 *   insert   the misses of a window are stored; where several map to one
 *            slot, the largest key wins; an insert replaces the slot's entry.
 * The content after every window depends only on the windows' keys and
 * results, never on thread timing.  Stored rows are those of the corpus the
 * window was scored against: call hs_cache_reset when the corpus changes.
 * Calls on one store must not overlap (same stream, or ordered by events). */

/* *bytes = size of the store buffer for `capacity` entries of the plan's k. */
hs_status hs_cache_bytes(const hs_plan *plan, int64_t capacity, size_t *bytes);

/* Empties the store (every slot invalid).  Needed once before first use. */
hs_status hs_cache_reset(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                         void *stream);

/* Looks up the window's distinct keys (hs_dedup's unique_keys / first_index,
 * with n_unique / n_unique_dev as for hs_score_topk):
 *   topk_score/index [n_u x k] out: rows of the hits are filled with the
 *                    stored result; rows of the misses are left untouched
 *   miss_pos   [n_u] int32 out: -1 for a hit, else the miss's position in
 *              the miss list (misses numbered in ascending key order)
 *   miss_first [n_u] int32 out: entry p (< n_miss) = first_index of miss p,
 *              i.e. the request whose query row represents it (entries from
 *              n_miss on are unspecified)
 *   n_miss_dev int64 device out: number of misses n_m
 * The misses are then scored as a window of n_m distinct nodes (query rows
 * gathered through miss_first, hs_score_topk with n_unique_dev = n_miss_dev)
 * and their rows put back in place with hs_scatter(index = miss_pos), which
 * leaves the hit rows alone. */
hs_status hs_cache_lookup(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                          const int64_t *unique_keys, const int32_t *first_index,
                          int64_t n_unique, const int64_t *n_unique_dev, float *topk_score,
                          int32_t *topk_index, int32_t *miss_pos, int32_t *miss_first,
                          int64_t *n_miss_dev, void *stream);

/* Stores the rows of the window's misses (miss_pos from hs_cache_lookup on
 * the same store, no other call on it in between; topk_score/index are the
 * window's complete [n_u x k] rows). */
hs_status hs_cache_insert(const hs_plan *plan, void *cache, size_t cache_bytes, int64_t capacity,
                          const int64_t *unique_keys, const int32_t *miss_pos, int64_t n_unique,
                          const int64_t *n_unique_dev, const float *topk_score,
                          const int32_t *topk_index, void *stream);

/* Node signatures (Eq. 2; SHA-256 as in the paper's prototype, Sec. 4.1).
 * Sig(v) = SHA-256 of the message, all integers little-endian,
 *     le32(tau_v) | le32(|Theta|) | Theta | le32(|D|) | D | le32(m) |
 *     Sig(u_1) | ... | Sig(u_m)
 * with tau_v the operator type, Theta the bytes of the parameters that affect
 * the node's result (e.g. Top-K), D the node's input text (normalised when
 * HS_SIG_NORMALIZE_TEXT is set: ASCII A-Z folded to a-z, every run of ASCII
 * whitespace -- space, \t, \n, \v, \f, \r -- replaced by one space, leading
 * and trailing whitespace dropped, all other bytes unchanged) and Sig(u_j) the
 * 32-byte digests of the node's m predecessors in the given order.  The key
 * that feeds hs_dedup is the digest's first 8 bytes read big-endian as a
 * signed int64.  One call hashes nodes [first, first + count); their
 * predecessors must have been hashed by earlier calls (ids < first), so a DAG
 * is hashed one topological level per call on one stream.
 * The struct is read on the host during the call; its pointers are device
 * addresses. */
typedef struct {
    const uint32_t *op_type;   /* [n_nodes] tau_v */
    const uint8_t *params;     /* Theta bytes of all nodes, concatenated */
    const int64_t *param_off;  /* [n_nodes + 1]: node i's Theta is
                                  params[param_off[i], param_off[i+1]); NULL = none */
    int64_t param_bytes;       /* bytes in params, 0 <= . <= 2^32 - 16 */
    const uint8_t *text;       /* D bytes of all nodes, concatenated */
    const int64_t *text_off;   /* [n_nodes + 1] as param_off; NULL = empty texts */
    int64_t text_bytes;        /* bytes in text, 0 <= . <= 2^32 - 16 */
    const int32_t *pred_off;   /* [n_nodes + 1] into pred_idx; NULL = no predecessors */
    const int32_t *pred_idx;   /* [pred_count] predecessor node ids, ordered */
    int64_t pred_count;        /* 0 <= . <= 2^31 - 1 */
    int64_t n_nodes;           /* 0 <= . <= 2^27 */
} hs_sig_nodes;

#define HS_SIG_NORMALIZE_TEXT 1

/*   digest  [n_nodes x 32] bytes device, 16-byte aligned: rows < first are
 *           read (predecessor digests), rows [first, first + count) written
 *   keys    [n_nodes] int64 device out, may be NULL: entries
 *           [first, first + count) written
 * Offsets are clamped to their buffers (a range past the end is cut there, a
 * reversed range is empty); a predecessor id outside [0, first) is hashed as
 * 32 zero bytes.  Bit-exact and deterministic. */
hs_status hs_signature(const hs_sig_nodes *nodes, int64_t first, int64_t count, int32_t flags,
                       uint8_t *digest, int64_t *keys, void *stream);

/* Reuse-driven priorities of the fused nodes (Eq. 3) and their order in the
 * ready queue (Eq. 7; Algorithm 1, phase 2), from hs_dedup's groups:
 *   inverse, first_index  hs_dedup outputs ([R] and [n_u] int32 device)
 *   n_unique / n_unique_dev  as for hs_score_topk
 *   phi      [R] fp32 device: contribution phi_v of each logical node (Eq. 5,
 *            computed upstream); clamped to [0, 2^16), NaN counts as 0
 *   s_hat    [R] fp32 device: remaining-time estimate S_q of each node's
 *            query (Eq. 4, computed upstream), >= 0
 *   heavy    [R] uint8 device, may be NULL (all 0): heavy-node flag y_v
 *   alpha, gamma, delta, eps  the weights of Eq. 7 (finite; eps > 0)
 *   phi_fused [n_u] fp64 device out, may be NULL: phi* of Eq. 3 = the sum of
 *            the group's phi_v, each truncated to a multiple of 2^-24 first;
 *            exact (independent of the order of the additions) and rounded
 *            once to fp64, for groups whose sum stays below 2^39
 *   pi       [n_u] fp64 device out, may be NULL:
 *            ((alpha / (s_hat[s] + eps)) + gamma * phi*) + delta * heavy[s],
 *            each operation rounded to nearest, s = first_index[g] (the
 *            surviving node, to which the merged nodes' edges are redirected)
 *   order    [n_u] int32 device out: the fused nodes by pi descending, equal
 *            pi by ascending group (-0 as +0)
 *   ws       the plan's workspace (hs_merge_plan's size covers this call)
 * Bit-exact and deterministic. */
hs_status hs_priority(const hs_plan *plan, const int32_t *inverse, const int32_t *first_index,
                      int64_t n_unique, const int64_t *n_unique_dev, const float *phi,
                      const float *s_hat, const uint8_t *heavy, double alpha, double gamma,
                      double delta, double eps, double *phi_fused, double *pi, int32_t *order,
                      void *ws, size_t ws_bytes, void *stream);

const char *hs_status_string(hs_status s);
const char *hs_last_error(void);
int32_t hs_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HS_MERGE_H */
