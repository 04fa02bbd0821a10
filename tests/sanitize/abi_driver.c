/* Host sanitizer run of the C ABI's argument validation (api.cpp built with
 * host-only launcher stubs, -fsanitize=address,undefined): every entry point
 * with bad arguments returns its documented status, leaves a message and
 * launches nothing; with good arguments it validates and reaches its
 * launchers.  Device pointers are fake addresses that are never
 * dereferenced.  Exit status 0 = all checks passed. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "hs_merge.h"

extern int hs_stub_launches;
static int fails = 0;
#define CHECK(c)                                                            \
    do {                                                                    \
        if (!(c)) {                                                         \
            fprintf(stderr, "check failed at line %d: %s (last error: %s)\n", __LINE__, #c, \
                    hs_last_error());                                       \
            ++fails;                                                        \
        }                                                                   \
    } while (0)

#define P(x) ((void *)(uintptr_t)(x))
static const uintptr_t F = 0x10000000;   /* fake, 256-byte aligned */

/* status s, a message, and no launch */
#define REJECT(call, s)                                                     \
    do {                                                                    \
        int before = hs_stub_launches;                                      \
        CHECK((call) == (s));                                               \
        CHECK(hs_last_error()[0] != 0);                                     \
        CHECK(hs_stub_launches == before);                                  \
    } while (0)
#define ACCEPT(call, nlaunch)                                               \
    do {                                                                    \
        int before = hs_stub_launches;                                      \
        CHECK((call) == HS_OK);                                             \
        CHECK(hs_stub_launches == before + (nlaunch));                      \
    } while (0)

static hs_plan *plan_of(int64_t R, int64_t d, int64_t N, int k, int qd, int cd, int64_t cap,
                        int64_t W, const int64_t *off, size_t *ws) {
    hs_merge_desc desc;
    memset(&desc, 0, sizeof(desc));
    desc.n_requests = R;
    desc.dim = d;
    desc.n_corpus = N;
    desc.k = k;
    desc.query_dtype = qd;
    desc.corpus_dtype = cd;
    desc.max_unique = cap;
    desc.n_workflows = W;
    desc.workflow_offsets = off;
    hs_plan *p = NULL;
    return hs_merge_plan(&desc, &p, ws) == HS_OK ? p : NULL;
}

static hs_plan *plan_flags(int64_t R, int64_t d, int64_t N, int k, int qd, int cd, int32_t flags,
                           size_t *ws) {
    hs_merge_desc desc;
    memset(&desc, 0, sizeof(desc));
    desc.n_requests = R;
    desc.dim = d;
    desc.n_corpus = N;
    desc.k = k;
    desc.query_dtype = qd;
    desc.corpus_dtype = cd;
    desc.flags = flags;
    desc.n_workflows = 1;
    hs_plan *p = NULL;
    return hs_merge_plan(&desc, &p, ws) == HS_OK ? p : NULL;
}

int main(void) {
    size_t ws = 0;
    CHECK(hs_abi_version() == HS_ABI_VERSION);
    CHECK(strcmp(hs_status_string(HS_ERR_WORKSPACE), "HS_ERR_WORKSPACE") == 0);

    /* plans */
    hs_merge_desc bad;
    memset(&bad, 0, sizeof(bad));
    hs_plan *p = NULL;
    REJECT(hs_merge_plan(NULL, &p, &ws), HS_ERR_INVALID_ARG);
    bad.n_requests = 8; bad.dim = 8; bad.n_corpus = 10; bad.k = 3;
    bad.query_dtype = HS_BF16; bad.corpus_dtype = HS_BF16; bad.n_workflows = 0;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_INVALID_ARG);           /* W = 0 */
    bad.n_workflows = 3;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_INVALID_ARG);           /* 3 does not divide 8 */
    int64_t off_bad[4] = {0, 6, 4, 8}, off_ok[4] = {0, 0, 5, 8};
    bad.workflow_offsets = off_bad;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_INVALID_ARG);
    bad.workflow_offsets = off_ok;
    bad.dim = 12;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_UNSUPPORTED);           /* bf16 needs d % 8 */
    bad.dim = 8; bad.k = 0;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_INVALID_ARG);
    bad.k = 3; bad.flags = 4;
    REJECT(hs_merge_plan(&bad, &p, &ws), HS_ERR_INVALID_ARG);
    bad.flags = 0;
    CHECK(hs_merge_plan(&bad, &p, &ws) == HS_OK && p);
    int64_t first = -1, count = -1;
    CHECK(hs_workflow_rows(p, 2, &first, &count) == HS_OK && first == 5 && count == 3);
    REJECT(hs_workflow_rows(p, 3, &first, &count), HS_ERR_INVALID_ARG);
    hs_plan_destroy(p);

    /* a 1M-row window: R = 2048, d = 768, k = 10, 64 workflows */
    hs_plan *w = plan_of(2048, 768, 1000000, 10, HS_BF16, HS_BF16, 0, 64, NULL, &ws);
    CHECK(w != NULL && ws > 0);
    if (!w) return 1;
    int64_t host_nu = 0;
    REJECT(hs_dedup(w, P(F), P(F), P(F), P(F), P(F), NULL, NULL, P(F), ws, NULL),
           HS_ERR_INVALID_ARG);
    REJECT(hs_dedup(w, P(F + 4), P(F), P(F), P(F), P(F), P(F), NULL, P(F), ws, NULL),
           HS_ERR_ALIGNMENT);
    ACCEPT(hs_dedup(w, P(F), P(F), P(F), NULL, P(F), P(F), NULL, P(F), ws, NULL), 1);
    (void)host_nu;
    REJECT(hs_score_topk(w, P(F), 4096, NULL, P(F), NULL, P(F), P(F), P(F), ws, NULL),
           HS_ERR_INVALID_ARG);
    REJECT(hs_score_topk(w, P(F), -1, NULL, P(F), NULL, P(F), P(F), P(F), ws, NULL),
           HS_ERR_INVALID_ARG);
    REJECT(hs_score_topk(w, P(F), 10, NULL, P(F), NULL, P(F), P(F), P(F), ws - 1, NULL),
           HS_ERR_WORKSPACE);
    REJECT(hs_score_topk(w, P(F), 10, NULL, P(F + 8), NULL, P(F), P(F), P(F), ws, NULL),
           HS_ERR_ALIGNMENT);
    ACCEPT(hs_score_topk(w, P(F), 10, NULL, P(F), NULL, P(F), P(F), P(F), ws, NULL), 2);
    ACCEPT(hs_score_partial(w, P(F), -1, P(F), P(F), NULL, P(F), ws, NULL), 1);
    ACCEPT(hs_topk_merge(w, -1, P(F), P(F), P(F), P(F), ws, NULL), 1);
    /* tiled corpus layout */
    size_t tb = 0;
    CHECK(hs_corpus_tiled_bytes(w, &tb) == HS_OK && tb == (size_t)2605 * 384 * 768 * 2);
    REJECT(hs_corpus_tiled_bytes(w, NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_tile_corpus(w, NULL, P(F + (1ull << 33)), tb, NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_tile_corpus(w, P(F), P(F + (1ull << 33)), tb - 16, NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_tile_corpus(w, P(F), P(F + 4096), tb, NULL), HS_ERR_INVALID_ARG);  /* overlap */
    REJECT(hs_tile_corpus(w, P(F + 8), P(F + (1ull << 33)), tb, NULL), HS_ERR_ALIGNMENT);
    ACCEPT(hs_tile_corpus(w, P(F), P(F + (1ull << 33)), tb, NULL), 1);
    hs_plan *wt = plan_flags(2048, 768, 1000000, 10, HS_BF16, HS_BF16, HS_FLAG_TILED_CORPUS, &ws);
    CHECK(wt != NULL);
    if (wt) {
      ACCEPT(hs_score_topk(wt, P(F), 10, NULL, P(F), NULL, P(F), P(F), P(F), ws, NULL), 2);
      hs_plan_destroy(wt);
    }
    CHECK(plan_flags(64, 768, 1000, 10, HS_F32, HS_F32, HS_FLAG_TILED_CORPUS, &ws) == NULL);
    /* the allocation-free variant validates, then finds no GPU here */
    REJECT(hs_score_topk_noalloc(w, P(F), 4096, NULL, P(F), NULL, P(F), P(F), NULL),
           HS_ERR_INVALID_ARG);
    CHECK(hs_score_topk_noalloc(w, P(F), 10, NULL, P(F), NULL, P(F), P(F), NULL) ==
          HS_ERR_DEVICE);
    REJECT(hs_scatter(P(F), 10, 6, P(F), 0, 5, NULL, P(F), NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_scatter(P(F), 10, 8, P(F + 4), 1, 5, NULL, P(F), NULL), HS_ERR_ALIGNMENT);
    ACCEPT(hs_scatter(P(F), 10, 8, P(F), 1, 5, P(F), P(F), NULL), 1);
    ACCEPT(hs_scatter(P(F), 10, 8, P(F), 1, 0, NULL, P(F), NULL), 0);
    REJECT(hs_deliver(w, P(F), P(F), -1, P(F), P(F), P(F), NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_deliver(w, P(F), NULL, 5, P(F), P(F), P(F), NULL), HS_ERR_INVALID_ARG);
    ACCEPT(hs_deliver(w, P(F), P(F), 5, P(F), P(F), P(F), NULL), 1);
    size_t cb = 0;
    REJECT(hs_cache_bytes(w, 3, &cb), HS_ERR_INVALID_ARG);
    CHECK(hs_cache_bytes(w, 1024, &cb) == HS_OK && cb > 0);
    REJECT(hs_cache_reset(w, P(F), cb - 1, 1024, NULL), HS_ERR_WORKSPACE);
    ACCEPT(hs_cache_reset(w, P(F), cb, 1024, NULL), 1);
    REJECT(hs_cache_lookup(w, P(F), cb, 1024, P(F), P(F), 10, NULL, P(F), P(F), P(F), P(F),
                           NULL, NULL), HS_ERR_INVALID_ARG);
    ACCEPT(hs_cache_lookup(w, P(F), cb, 1024, P(F), P(F), 10, NULL, P(F), P(F), P(F), P(F),
                           P(F), NULL), 1);
    ACCEPT(hs_cache_insert(w, P(F), cb, 1024, P(F), P(F), -1, P(F), P(F), P(F), NULL), 1);
    REJECT(hs_priority(w, P(F), P(F), 10, NULL, P(F), P(F), NULL, 1.0, 1.0, 0.0, 0.0, NULL,
                       NULL, P(F), P(F), ws, NULL), HS_ERR_INVALID_ARG);   /* eps = 0 */
    ACCEPT(hs_priority(w, P(F), P(F), 10, NULL, P(F), P(F), NULL, 1.0, 1.0, 0.0, 0.5, NULL,
                       NULL, P(F), P(F), ws, NULL), 1);
    hs_sig_nodes nd;
    memset(&nd, 0, sizeof(nd));
    nd.op_type = P(F);
    nd.n_nodes = 10;
    REJECT(hs_signature(&nd, 5, 6, 0, P(F), NULL, NULL), HS_ERR_INVALID_ARG);
    REJECT(hs_signature(&nd, 0, 4, 0, P(F + 8), NULL, NULL), HS_ERR_ALIGNMENT);
    ACCEPT(hs_signature(&nd, 0, 4, HS_SIG_NORMALIZE_TEXT, P(F), P(F), NULL), 1);
    hs_plan_destroy(w);

    if (fails) fprintf(stderr, "%d checks failed\n", fails);
    else printf("C ABI validation: all checks passed\n");
    return fails ? 1 : 0;
}
