/*
 * Seeded synthetic inputs for the merged-retrieval workloads.
 *
 * This file holds NO arithmetic of the method (no deduplication, scoring or
 * selection).  It only produces inputs: request keys drawn from a Zipf law,
 * unit-norm Gaussian vectors, and their storage encodings (fp32, bf16 and
 * OCP fp8 e4m3 with a per-row fp32 scale).  Both the oracle and the GPU
 * library consume the bytes written here.
 *
 * Every value is a pure function of (seed, stream, counter): a SplitMix64
 * counter generator (Steele, Lea & Flood, OOPSLA 2014) feeds Box-Muller
 * (1958).  Output bytes therefore do not depend on the thread count, and any
 * row can be regenerated on its own.
 *
 * Built with gcc into libsynth.so; driven from synth/__init__.py.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ull

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Base state of one named stream of one seed. */
uint64_t syn_stream_base(uint64_t seed, uint64_t stream) {
    return mix64(seed + GAMMA) ^ mix64(stream * GAMMA + 0x632BE59BD9B4E019ull);
}

/* Draw number `ctr` of the stream whose base is `base` (the SplitMix64
 * sequence started at `base`). */
static inline uint64_t draw(uint64_t base, uint64_t ctr) {
    return mix64(base + (ctr + 1) * GAMMA);
}

uint64_t syn_draw(uint64_t base, uint64_t ctr) { return draw(base, ctr); }

/* Uniform in the open interval (0, 1) from the top 53 bits. */
static inline double unif(uint64_t u) {
    return ((double)(u >> 11) + 0.5) * 0x1.0p-53;
}

/* Round an fp32 value to bf16 (round to nearest, ties to even).  Inputs are
 * finite. */
static inline uint16_t f32_to_bf16(float f) {
    uint32_t b;
    memcpy(&b, &f, 4);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

uint16_t syn_f32_to_bf16(float f) { return f32_to_bf16(f); }

/* Encode a finite double as OCP fp8 e4m3 ("fn": bias 7, no infinities, the
 * all-ones pattern is NaN, largest finite 448), rounding to nearest with ties
 * to even.  Magnitudes at or above 448 saturate to 448. */
uint8_t syn_e4m3_encode(double v) {
    uint8_t sign = signbit(v) ? 0x80 : 0x00;
    double a = fabs(v);
    if (a == 0.0) return sign;
    if (a >= 448.0) return sign | 0x7E;
    int e;
    frexp(a, &e);
    int E = e - 1;               /* a in [2^E, 2^(E+1)) */
    if (E < -6) E = -6;          /* subnormal binade shares quantum 2^-9 */
    double q = ldexp(1.0, E - 3);
    double r = nearbyint(a / q) * q;  /* a/q is exact: q is a power of two */
    if (r == 0.0) return sign;
    if (r >= 448.0) return sign | 0x7E;
    int e2;
    frexp(r, &e2);
    int E2 = e2 - 1;
    if (E2 < -6) return sign | (uint8_t)(r / ldexp(1.0, -9));
    int mant = (int)(r / ldexp(1.0, E2 - 3)) - 8;
    return sign | (uint8_t)(((E2 + 7) << 3) | mant);
}

/* ---- unit-norm Gaussian rows ------------------------------------------- */

enum { ENC_F32 = 0, ENC_BF16 = 1, ENC_FP8 = 2 };

typedef struct {
    uint64_t base;      /* stream base */
    const int64_t *row_ids; /* which logical rows to generate (NULL: first + i) */
    int64_t first;
    int64_t n_rows;
    int64_t dim;
    int enc;
    void *out;          /* n_rows x dim, encoding `enc` */
    float *scale;       /* fp8 only: n_rows */
    int64_t lo, hi;     /* this worker's slice of [0, n_rows) */
} rows_job;

static void gen_one_row(uint64_t base, int64_t row, int64_t dim, double *x) {
    int64_t pairs = dim / 2;
    double ss = 0.0;
    for (int64_t p = 0; p < pairs; ++p) {
        uint64_t c = (uint64_t)(row * pairs + p) * 2u;
        double u1 = unif(draw(base, c));
        double u2 = unif(draw(base, c + 1));
        double rr = sqrt(-2.0 * log(u1));
        double th = 6.283185307179586476925286766559 * u2;
        x[2 * p] = rr * cos(th);
        x[2 * p + 1] = rr * sin(th);
        ss += x[2 * p] * x[2 * p] + x[2 * p + 1] * x[2 * p + 1];
    }
    double inv = 1.0 / sqrt(ss);
    for (int64_t j = 0; j < dim; ++j) x[j] *= inv;
}

static void *rows_worker(void *arg) {
    rows_job *jb = (rows_job *)arg;
    double *x = (double *)malloc(sizeof(double) * (size_t)jb->dim);
    float *f = (float *)malloc(sizeof(float) * (size_t)jb->dim);
    for (int64_t i = jb->lo; i < jb->hi; ++i) {
        int64_t row = jb->row_ids ? jb->row_ids[i] : jb->first + i;
        gen_one_row(jb->base, row, jb->dim, x);
        for (int64_t j = 0; j < jb->dim; ++j) f[j] = (float)x[j];
        size_t off = (size_t)i * (size_t)jb->dim;
        if (jb->enc == ENC_F32) {
            memcpy((float *)jb->out + off, f, sizeof(float) * (size_t)jb->dim);
        } else if (jb->enc == ENC_BF16) {
            uint16_t *o = (uint16_t *)jb->out + off;
            for (int64_t j = 0; j < jb->dim; ++j) o[j] = f32_to_bf16(f[j]);
        } else {
            float amax = 0.0f;
            for (int64_t j = 0; j < jb->dim; ++j) {
                float a = fabsf(f[j]);
                if (a > amax) amax = a;
            }
            float s = amax > 0.0f ? amax / 448.0f : 1.0f;
            jb->scale[i] = s;
            uint8_t *o = (uint8_t *)jb->out + off;
            for (int64_t j = 0; j < jb->dim; ++j)
                o[j] = syn_e4m3_encode((double)f[j] / (double)s);
        }
    }
    free(x);
    free(f);
    return NULL;
}

/* Generate rows of a unit-norm Gaussian matrix.  Row `row_ids[i]` (or
 * `first + i` when row_ids is NULL) goes to output row i.  dim must be even.
 * Returns 0 on success. */
int syn_gaussian_rows(uint64_t seed, uint64_t stream, const int64_t *row_ids,
                      int64_t first, int64_t n_rows, int64_t dim, int enc,
                      void *out, float *scale, int n_threads) {
    if (dim <= 0 || (dim & 1) || n_rows < 0 || !out) return -1;
    if (enc == ENC_FP8 && !scale) return -1;
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    if (n_rows < n_threads) n_threads = n_rows > 0 ? (int)n_rows : 1;
    pthread_t th[256];
    rows_job jobs[256];
    uint64_t base = syn_stream_base(seed, stream);
    for (int t = 0; t < n_threads; ++t) {
        rows_job *jb = &jobs[t];
        jb->base = base;
        jb->row_ids = row_ids;
        jb->first = first;
        jb->n_rows = n_rows;
        jb->dim = dim;
        jb->enc = enc;
        jb->out = out;
        jb->scale = scale;
        jb->lo = n_rows * t / n_threads;
        jb->hi = n_rows * (t + 1) / n_threads;
    }
    for (int t = 1; t < n_threads; ++t) pthread_create(&th[t], NULL, rows_worker, &jobs[t]);
    rows_worker(&jobs[0]);
    for (int t = 1; t < n_threads; ++t) pthread_join(th[t], NULL);
    return 0;
}

/* ---- Zipf request streams ------------------------------------------------ */

/* Seeded Fisher-Yates permutation of [0, m). */
int syn_permutation(uint64_t seed, uint64_t stream, int64_t m, int64_t *perm) {
    if (m < 0 || !perm) return -1;
    uint64_t base = syn_stream_base(seed, stream);
    for (int64_t i = 0; i < m; ++i) perm[i] = i;
    for (int64_t i = m - 1; i > 0; --i) {
        int64_t j = (int64_t)(draw(base, (uint64_t)i) % (uint64_t)(i + 1));
        int64_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
    return 0;
}

/* Draw n ranks in [0, m) with P(rank r) proportional to (r+1)^-s, by inverse
 * CDF (binary search in an fp64 cumulative table). */
int syn_zipf_ranks(uint64_t seed, uint64_t stream, int64_t m, double s,
                   int64_t n, int64_t *ranks) {
    if (m <= 0 || n < 0 || !ranks) return -1;
    double *cdf = (double *)malloc(sizeof(double) * (size_t)m);
    if (!cdf) return -2;
    double acc = 0.0;
    for (int64_t r = 0; r < m; ++r) {
        acc += pow((double)(r + 1), -s);
        cdf[r] = acc;
    }
    uint64_t base = syn_stream_base(seed, stream);
    for (int64_t i = 0; i < n; ++i) {
        double u = unif(draw(base, (uint64_t)i)) * acc;
        int64_t lo = 0, hi = m - 1;
        while (lo < hi) {
            int64_t mid = lo + (hi - lo) / 2;
            if (cdf[mid] >= u) hi = mid; else lo = mid + 1;
        }
        ranks[i] = lo;
    }
    free(cdf);
    return 0;
}
