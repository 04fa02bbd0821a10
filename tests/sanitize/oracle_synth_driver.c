/* Host sanitizer run of the oracle (oracle/oracle.c) and the input generator
 * (synth/gen.c): every exported function on small inputs, including edge
 * sizes (R = 0, k > N, one thread, more threads than rows), built with
 * -fsanitize=address,undefined.  Exit status 0 = no failed check (the
 * sanitizers abort on their own findings). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double or_e4m3_decode(uint8_t code);
double or_bf16_decode(uint16_t bits);
int or_dedup(const int64_t *keys, int64_t R, int64_t *unique_keys, int32_t *first_index,
             int32_t *counts, int32_t *inverse, int64_t *n_unique);
int or_gather_rows(const void *src, int64_t src_rows, int64_t row_bytes, const void *index,
                   int index_is_i64, int64_t n_out, void *dst);
int or_topk_exact(const void *Q, int q_enc, int64_t n_sel, const int64_t *q_rows, const void *C,
                  int c_enc, const float *scale, int64_t N, int64_t d, int64_t kk,
                  double *best_score, int64_t *best_index, int threads);
int or_score_pairs(const void *Q, int q_enc, const void *C, int c_enc, const float *scale,
                   int64_t d, int64_t n_pairs, const int64_t *q_idx, const int64_t *c_idx,
                   double *out, int threads);
int or_merge_retrieval(const int64_t *keys, int64_t R, const void *Q_req, int q_enc,
                       const void *C, int c_enc, const float *scale, int64_t N, int64_t d,
                       int64_t k, int64_t n_sel, const int64_t *u_sel, int64_t *unique_keys,
                       int32_t *first_index, int32_t *counts, int32_t *inverse,
                       int64_t *n_unique, float *u_score, int32_t *u_index, float *out_score,
                       int32_t *out_index, int threads);
uint64_t syn_stream_base(uint64_t seed, uint64_t stream);
uint64_t syn_draw(uint64_t base, uint64_t ctr);
uint16_t syn_f32_to_bf16(float f);
uint8_t syn_e4m3_encode(double v);
int syn_gaussian_rows(uint64_t seed, uint64_t stream, const int64_t *row_ids, int64_t first,
                      int64_t n_rows, int64_t dim, int enc, void *out, float *scale,
                      int n_threads);
int syn_permutation(uint64_t seed, uint64_t stream, int64_t m, int64_t *perm);
int syn_zipf_ranks(uint64_t seed, uint64_t stream, int64_t m, double s, int64_t n,
                   int64_t *ranks);

static int fails = 0;
#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++fails;                                               \
        }                                                          \
    } while (0)

int main(void) {
    /* decoders */
    for (int c = 0; c < 256; ++c) (void)or_e4m3_decode((uint8_t)c);
    CHECK(or_e4m3_decode(0x7E) == 448.0 && isnan(or_e4m3_decode(0x7F)));
    CHECK(or_bf16_decode(0x3F80) == 1.0);
    CHECK(syn_f32_to_bf16(1.0f) == 0x3F80 && syn_e4m3_encode(448.0) == 0x7E);

    /* generator: every encoding, explicit row ids, more threads than rows */
    const int64_t d = 24, N = 37, nq = 5;
    uint16_t *cb = malloc(sizeof(uint16_t) * N * d);
    float *cf = malloc(sizeof(float) * N * d);
    uint8_t *c8 = malloc((size_t)(N * d));
    float *sc = malloc(sizeof(float) * N);
    uint16_t *qb = malloc(sizeof(uint16_t) * nq * d);
    int64_t ids[5] = {3, 99, 0, 3, 7};
    CHECK(syn_gaussian_rows(1, 2, NULL, 0, N, d, 1, cb, NULL, 64) == 0);
    CHECK(syn_gaussian_rows(1, 2, NULL, 0, N, d, 0, cf, NULL, 1) == 0);
    CHECK(syn_gaussian_rows(1, 2, NULL, 0, N, d, 2, c8, sc, 3) == 0);
    CHECK(syn_gaussian_rows(1, 3, ids, 0, nq, d, 1, qb, NULL, 2) == 0);
    CHECK(syn_gaussian_rows(1, 3, NULL, 0, 0, d, 1, qb, NULL, 4) == 0);       /* no rows */
    CHECK(syn_gaussian_rows(1, 3, NULL, 0, 4, 7, 1, qb, NULL, 4) == -1);      /* odd dim */
    CHECK(memcmp(qb, qb + 3 * d, sizeof(uint16_t) * d) == 0);                /* same id */
    int64_t perm[50], ranks[200];
    CHECK(syn_permutation(9, 1, 50, perm) == 0 && syn_permutation(9, 1, 0, perm) == 0);
    CHECK(syn_zipf_ranks(9, 2, 17, 1.1, 200, ranks) == 0);
    for (int i = 0; i < 200; ++i) CHECK(ranks[i] >= 0 && ranks[i] < 17);
    (void)syn_draw(syn_stream_base(1, 2), 5);

    /* dedup: empty, extremes */
    int64_t keys[12] = {5, -1, INT64_MIN, 5, INT64_MAX, -1, 0, 5, 9, INT64_MIN, 0, 2};
    int64_t uk[12], nu = -1;
    int32_t fi[12], ct[12], inv[12];
    CHECK(or_dedup(keys, 0, uk, fi, ct, inv, &nu) == 0 && nu == 0);
    CHECK(or_dedup(keys, 12, uk, fi, ct, inv, &nu) == 0 && nu == 7);
    CHECK(or_dedup(keys, 12, uk, fi, NULL, inv, &nu) == 0);

    /* gather: in range, and an index out of range is refused */
    uint16_t g[5 * 24];
    int32_t gi[5] = {0, 36, 4, 4, 1};
    CHECK(or_gather_rows(cb, N, d * 2, gi, 0, 5, g) == 0);
    gi[2] = 37;
    CHECK(or_gather_rows(cb, N, d * 2, gi, 0, 5, g) == -1);

    /* top-k: k > N pads, selected rows, fp8 with scales, 1 and 64 threads */
    double bs[5 * 40];
    int64_t bi[5 * 40], sel[2] = {4, 1};
    CHECK(or_topk_exact(qb, 1, nq, NULL, cb, 1, NULL, N, d, 40, bs, bi, 64) == 0);
    CHECK(bi[39] == -1 && isinf(bs[39]));
    CHECK(or_topk_exact(qb, 1, 2, sel, c8, 2, sc, N, d, 7, bs, bi, 1) == 0);
    CHECK(or_topk_exact(cf, 0, 3, NULL, cf, 0, NULL, N, d, 1, bs, bi, 5) == 0 && bi[0] == 0);
    CHECK(or_topk_exact(qb, 1, 0, NULL, cb, 1, NULL, N, d, 3, bs, bi, 2) == 0);
    int64_t qi[3] = {0, 4, 2}, ci[3] = {36, 0, 5};
    double sp[3];
    CHECK(or_score_pairs(qb, 1, c8, 2, sc, d, 3, qi, ci, sp, 2) == 0);

    /* merged retrieval, all and a selection */
    int64_t rk[5] = {11, 22, 11, 33, 22};
    float us[5 * 6], os[5 * 6];
    int32_t ui[5 * 6], oi[5 * 6];
    CHECK(or_merge_retrieval(rk, 5, qb, 1, cb, 1, NULL, N, d, 6, 0, NULL, uk, fi, ct, inv, &nu,
                             us, ui, os, oi, 3) == 0 && nu == 3);
    int64_t usel[1] = {2};
    CHECK(or_merge_retrieval(rk, 5, qb, 1, cb, 1, NULL, N, d, 6, 1, usel, uk, fi, ct, inv, &nu,
                             us, ui, os, oi, 1) == 0);

    free(cb); free(cf); free(c8); free(sc); free(qb);
    if (fails) fprintf(stderr, "%d checks failed\n", fails);
    else printf("oracle and generator: all checks passed\n");
    return fails ? 1 : 0;
}
