/*
 * ORACLE -- test infrastructure, not part of the product.
 *
 * A plain, slow, obviously correct CPU implementation of merged retrieval:
 * cross-workflow deduplication of retrieval nodes by signature, one exact
 * inner-product top-k per distinct node, and delivery of each result to every
 * node that carries the same signature.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it.  It shares no source with
 * the GPU library and includes no GPU headers.
 *
 * What it follows (HeraSys, Li et al.):
 *  - Sec. 3.3, Eq. (2): a node's semantic signature identifies computationally
 *    equivalent nodes; equal signatures have equal outputs.  Here the
 *    signature arrives as a 64-bit key per request.
 *  - Sec. 3.3 "Topological Fusion within Time Window": a duplicate node is
 *    removed, its downstream edges are redirected to the surviving node, and
 *    the survivor's output flows to every related query.  The survivor is the
 *    earliest request; `inverse` is the redirected edge; `counts` is the size
 *    of the merged set M(v*) of Eq. (3).
 *  - Sec. 4.1 workloads: vector retrieval returns the top-K chunks; Eq. (2)
 *    lists Top-K among the parameters of a retrieval node.  Retrieval here is
 *    exact inner product; ties go to the lower chunk index.
 *  - Appendix complexity analysis, Phase 1: redundancy elimination is a
 *    lookup in a global duplication map.  The oracle realises that map by
 *    sorting (key, request) pairs, which yields the same groups in canonical
 *    (ascending key) order.
 *
 * Arithmetic: every input element is widened exactly to double (fp32 and
 * bf16 widen exactly; OCP e4m3 codes are decoded from the format definition),
 * products of these are exact in double, and the d-term sums are accumulated
 * in double -- so each score is the exact value up to ~1e-16 relative.
 * Output scores are the doubles rounded to fp32.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_BF16 = 1, OR_FP8 = 2 };

/* ---- element decoding --------------------------------------------------- */

/* OCP 8-bit floating point, E4M3: 1 sign bit, 4 exponent bits (bias 7),
 * 3 mantissa bits.  Exponent field 0 is subnormal (m/8 * 2^-6).  There are no
 * infinities; exponent 15 with mantissa 7 is NaN, so 448 is the largest
 * finite magnitude. */
double or_e4m3_decode(uint8_t code) {
    int s = code >> 7;
    int e = (code >> 3) & 0xF;
    int m = code & 0x7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0)
        v = ldexp((double)m, -9);            /* (m/8) * 2^(1-7) */
    else
        v = ldexp((double)(8 + m), e - 10);  /* (1 + m/8) * 2^(e-7) */
    return s ? -v : v;
}

/* bfloat16 is the upper half of an IEEE binary32. */
static double bf16_value(uint16_t bits) {
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, 4);
    return (double)f;
}

double or_bf16_decode(uint16_t bits) { return bf16_value(bits); }

/* The 256 E4M3 values, tabulated once from or_e4m3_decode. */
static double e4m3_table[256];
static int e4m3_table_ready = 0;

static void init_tables(void) {
    if (e4m3_table_ready) return;
    for (int c = 0; c < 256; ++c) e4m3_table[c] = or_e4m3_decode((uint8_t)c);
    e4m3_table_ready = 1;
}

/* ---- step 1: deduplication ----------------------------------------------- */

typedef struct { int64_t key; int64_t idx; } kv;

static int kv_cmp(const void *a, const void *b) {
    const kv *x = (const kv *)a, *y = (const kv *)b;
    if (x->key != y->key) return x->key < y->key ? -1 : 1;
    if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
    return 0;
}

/* Group R requests by key.  unique_keys ascending (signed), first_index =
 * earliest request of each group, counts = group sizes, inverse[i] = group
 * of request i.  Returns 0, or -1 on bad arguments / allocation failure. */
int or_dedup(const int64_t *keys, int64_t R, int64_t *unique_keys,
             int32_t *first_index, int32_t *counts, int32_t *inverse,
             int64_t *n_unique) {
    if (R < 0 || !n_unique) return -1;
    *n_unique = 0;
    if (R == 0) return 0;
    kv *a = (kv *)malloc(sizeof(kv) * (size_t)R);
    if (!a) return -1;
    for (int64_t i = 0; i < R; ++i) { a[i].key = keys[i]; a[i].idx = i; }
    qsort(a, (size_t)R, sizeof(kv), kv_cmp);
    int64_t g = -1;
    for (int64_t i = 0; i < R; ++i) {
        if (i == 0 || a[i].key != a[i - 1].key) {
            ++g;
            unique_keys[g] = a[i].key;
            first_index[g] = (int32_t)a[i].idx;   /* smallest idx of the group */
            if (counts) counts[g] = 0;
        }
        if (counts) counts[g] += 1;
        inverse[a[i].idx] = (int32_t)g;
    }
    *n_unique = g + 1;
    free(a);
    return 0;
}

/* ---- steps 2 and 5: row gather ------------------------------------------- */

/* dst[i] = src[index[i]] for i < n_out (rows of row_bytes bytes).  Returns -1
 * if an index is out of [0, src_rows). */
int or_gather_rows(const void *src, int64_t src_rows, int64_t row_bytes,
                   const void *index, int index_is_i64, int64_t n_out, void *dst) {
    for (int64_t i = 0; i < n_out; ++i) {
        int64_t r = index_is_i64 ? ((const int64_t *)index)[i]
                                 : (int64_t)((const int32_t *)index)[i];
        if (r < 0 || r >= src_rows) return -1;
        memcpy((char *)dst + i * row_bytes, (const char *)src + r * row_bytes,
               (size_t)row_bytes);
    }
    return 0;
}

/* ---- steps 3 and 4: exact scores and top-k ------------------------------- */

/* Row r of a [rows x d] matrix in encoding enc, widened exactly to double. */
static void widen_row(const void *M, int enc, int64_t r, int64_t d, double *out) {
    const int64_t o = r * d;
    switch (enc) {
    case OR_F32:
        for (int64_t j = 0; j < d; ++j) out[j] = (double)((const float *)M)[o + j];
        break;
    case OR_BF16:
        for (int64_t j = 0; j < d; ++j) out[j] = bf16_value(((const uint16_t *)M)[o + j]);
        break;
    default:
        for (int64_t j = 0; j < d; ++j) out[j] = e4m3_table[((const uint8_t *)M)[o + j]];
        break;
    }
}

/* exact s(q, c) = scale_c * sum_j q[j] * C[c, j]  (scale_c = 1 unless fp8);
 * q is the query row already widened to double, crow is scratch for the
 * widened corpus row. */
static double score_row(const double *q, const void *C, int c_enc,
                        const float *scale, int64_t c, int64_t d, double *crow) {
    widen_row(C, c_enc, c, d, crow);
    double acc = 0.0;
    for (int64_t j = 0; j < d; ++j) acc += q[j] * crow[j];
    if (c_enc == OR_FP8) acc *= (double)scale[c];
    return acc;
}

/* (sa, ca) ranks before (sb, cb): higher score first, then lower index. */
static int better(double sa, int64_t ca, double sb, int64_t cb) {
    return sa > sb || (sa == sb && ca < cb);
}

/* Insert (s, c) into the sorted list bs/bi holding *filled of kk entries. */
static void list_insert(double *bs, int64_t *bi, int64_t kk, int64_t *filled, double s,
                        int64_t c) {
    if (*filled == kk && !better(s, c, bs[kk - 1], bi[kk - 1])) return;
    int64_t pos = *filled < kk ? *filled : kk - 1;   /* drop the last if full */
    while (pos > 0 && better(s, c, bs[pos - 1], bi[pos - 1])) {
        bs[pos] = bs[pos - 1];
        bi[pos] = bi[pos - 1];
        --pos;
    }
    bs[pos] = s;
    bi[pos] = c;
    if (*filled < kk) ++*filled;
}

/* For each selected query row q_rows[t] (or t when q_rows is NULL), the kk
 * best corpus rows by (score desc, index asc): one pass over all N corpus rows
 * in index order, each exact score offered to a sorted kk-entry list.  Outputs
 * [n_sel x kk]: best_score (double, exact), best_index (int64); slots beyond N
 * hold (-inf, -1).  Queries are independent; threads split the queries only,
 * so every list sees the rows exactly as in the definition. */
int or_topk_exact(const void *Q, int q_enc, int64_t n_sel, const int64_t *q_rows,
                  const void *C, int c_enc, const float *scale, int64_t N, int64_t d,
                  int64_t kk, double *best_score, int64_t *best_index, int threads) {
    if (n_sel < 0 || N < 0 || d <= 0 || kk <= 0) return -1;
    if (threads < 1) threads = 1;
    init_tables();
    int err = 0;
#pragma omp parallel for num_threads(threads) schedule(dynamic, 1)
    for (int64_t t = 0; t < n_sel; ++t) {
        int64_t q = q_rows ? q_rows[t] : t;
        double *bs = best_score + t * kk;
        int64_t *bi = best_index + t * kk;
        int64_t filled = 0;
        double *qv = (double *)malloc(sizeof(double) * 2 * (size_t)d);
        if (!qv) {
#pragma omp atomic write
            err = -1;
            continue;
        }
        widen_row(Q, q_enc, q, d, qv);
        for (int64_t c = 0; c < N; ++c)
            list_insert(bs, bi, kk, &filled, score_row(qv, C, c_enc, scale, c, d, qv + d), c);
        for (int64_t j = filled; j < kk; ++j) { bs[j] = -INFINITY; bi[j] = -1; }
        free(qv);
    }
    return err;
}

/* Exact scores of explicit (query row, corpus row) pairs. */
int or_score_pairs(const void *Q, int q_enc, const void *C, int c_enc,
                   const float *scale, int64_t d, int64_t n_pairs,
                   const int64_t *q_idx, const int64_t *c_idx, double *out, int threads) {
    if (threads < 1) threads = 1;
    init_tables();
    int err = 0;
#pragma omp parallel for num_threads(threads) schedule(static)
    for (int64_t p = 0; p < n_pairs; ++p) {
        double *qv = (double *)malloc(sizeof(double) * 2 * (size_t)d);
        if (!qv) {
#pragma omp atomic write
            err = -1;
            continue;
        }
        widen_row(Q, q_enc, q_idx[p], d, qv);
        out[p] = score_row(qv, C, c_enc, scale, c_idx[p], d, qv + d);
        free(qv);
    }
    return err;
}

/* ---- the whole merged retrieval ------------------------------------------- */

/* Steps 1-5 in order: dedup the R request keys, gather one representative
 * query row per distinct key, score and select top-k for the distinct rows
 * (only those listed in u_sel when u_sel is non-NULL: u_sel[t] is a distinct
 * position, and only requests whose group is selected get outputs), then
 * deliver each distinct result to all of its requests.
 *
 * Outputs: unique_keys/first_index/counts [R cap], inverse [R], n_unique;
 * u_score/u_index [n_sel x k] (the representative results, fp32 scores);
 * out_score/out_index [R x k] (per request; rows of unselected groups are
 * left untouched).  Returns 0 on success. */
int or_merge_retrieval(const int64_t *keys, int64_t R, const void *Q_req, int q_enc,
                       const void *C, int c_enc, const float *scale, int64_t N,
                       int64_t d, int64_t k, int64_t n_sel, const int64_t *u_sel,
                       int64_t *unique_keys, int32_t *first_index, int32_t *counts,
                       int32_t *inverse, int64_t *n_unique, float *u_score,
                       int32_t *u_index, float *out_score, int32_t *out_index,
                       int threads) {
    if (or_dedup(keys, R, unique_keys, first_index, counts, inverse, n_unique)) return -1;
    int64_t nu = *n_unique;
    if (!u_sel) n_sel = nu;
    int64_t qbytes = d * (q_enc == OR_F32 ? 4 : 2);
    /* representative rows, in the order of the selection */
    char *Qu = (char *)malloc((size_t)(n_sel > 0 ? n_sel : 1) * (size_t)qbytes);
    double *bs = (double *)malloc(sizeof(double) * (size_t)(n_sel > 0 ? n_sel : 1) * (size_t)k);
    int64_t *bi = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_sel > 0 ? n_sel : 1) * (size_t)k);
    int64_t *pos_of = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nu > 0 ? nu : 1));
    if (!Qu || !bs || !bi || !pos_of) { free(Qu); free(bs); free(bi); free(pos_of); return -1; }
    for (int64_t u = 0; u < nu; ++u) pos_of[u] = -1;
    for (int64_t t = 0; t < n_sel; ++t) {
        int64_t u = u_sel ? u_sel[t] : t;
        if (u < 0 || u >= nu) { free(Qu); free(bs); free(bi); free(pos_of); return -1; }
        pos_of[u] = t;
        memcpy(Qu + t * qbytes, (const char *)Q_req + (int64_t)first_index[u] * qbytes,
               (size_t)qbytes);
    }
    if (or_topk_exact(Qu, q_enc, n_sel, NULL, C, c_enc, scale, N, d, k, bs, bi, threads)) {
        free(Qu); free(bs); free(bi); free(pos_of);
        return -1;
    }
    for (int64_t t = 0; t < n_sel * k; ++t) {
        u_score[t] = (float)bs[t];
        u_index[t] = (int32_t)bi[t];
    }
    for (int64_t i = 0; i < R; ++i) {
        int64_t t = pos_of[inverse[i]];
        if (t < 0) continue;
        memcpy(out_score + i * k, u_score + t * k, sizeof(float) * (size_t)k);
        memcpy(out_index + i * k, u_index + t * k, sizeof(int32_t) * (size_t)k);
    }
    free(Qu); free(bs); free(bi); free(pos_of);
    return 0;
}
