// Steps 3 and 4: score every distinct query against the corpus and keep the
// k best rows per query.
//
// HeraSys runs one retrieval per fused node (Sec. 3.3 (I)) and batches ready
// nodes of the same type (Appendix A, batching constraint); a retrieval node's
// result is its Top-K chunks (Eq. 2 parameters; Sec. 4.1 workloads).  Here the
// batch is the n_u distinct queries and the retrieval is exact inner product.
//
// Phase 1 (this file, score_partial_*): one persistent kernel.  The grid is
// sized to the GPU; work items are (query tile of MQ, corpus slice) pairs, with
// S slices per query tile chosen on the device from n_u so the grid is filled
// whatever n_u turns out to be.  Items of one slice get consecutive logical
// ids and are mapped onto one XCD, so the query tiles that read the same
// corpus rows share that XCD's L2.  Per corpus tile of NC rows:
//   - bf16 / fp8 corpus: MFMA 32x32x16 bf16 with fp32 accumulation; the corpus
//     operand streams from HBM with 128-bit loads through double-buffered LDS;
//     fp8 e4m3 codes are widened to bf16 (exact) on the way into LDS and the
//     per-row scale is applied to the fp32 accumulator;
//   - fp32: plain VALU FMA tiles.
//   - epilogue: each lane compares its accumulators with the running k-th best
//     score of its query (held in registers); queries with a possible entrant
//     get their tile row scanned by one thread that keeps the query's k best
//     (score, row) keys of this slice.
// Phase 2 (topk_merge_kernel): per query, the S slice lists (S*k keys) are
// sorted and the first k are written out.
//
// Result keys order by (score desc, row asc), so ties always go to the lower
// corpus row, independently of which slice or lane saw them.
#include "common.h"

namespace hs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kMaxSK = 8192;        // bound on S*k (merge list length per query)
constexpr int kListLdsMaxK = 32;    // slice lists live in LDS up to this k
constexpr int kGridMax = 512;       // persistent grid never exceeds this

// MFMA path tiles
constexpr int kMQ = 128;            // queries per tile
constexpr int kNC = 128;            // corpus rows per tile
constexpr int kKC = 64;             // K per LDS stage
constexpr int kLda = kKC + 8;       // staged row stride (bf16 elements)
constexpr int kDumpLd = kNC + 4;    // dumped scores: floats per query row

// VALU (fp32) path tiles
constexpr int kVMQ = 64;
constexpr int kVNC = 64;
constexpr int kVKC = 32;
constexpr int kVLd = kVKC + 1;
constexpr int kVDumpLd = kVNC + 4;

struct ScoreArgs {
  const void *q;
  const void *corpus;
  const float *scale;
  int64_t N, d;
  int k;
  int64_t n_unique;
  const int64_t *n_unique_dev;
  int64_t cap;
  int grid;
  uint64_t *part;
};

__host__ __device__ __forceinline__ Split split_for(int64_t nu, int64_t N, int mq, int nc,
                                                   int grid, int k) {
  Split sp = make_split(nu, N, mq, nc, grid);
  int64_t smax = kMaxSK / k;
  if (smax < 1) smax = 1;
  if (sp.S > smax) sp.S = smax;
  return sp;
}

// Logical id of this workgroup: consecutive ids on one XCD (workgroups are
// dispatched round-robin over the 8 XCDs).
__device__ __forceinline__ int logical_wg(int grid) {
  int b = blockIdx.x;
  return (b & 7) * (grid >> 3) + (b >> 3);
}

// ---- per-query running lists (unsorted k keys + position of the minimum) ----

struct TileState {
  uint64_t *lmin;   // [MQ] smallest key in the list (0 while not full)
  int32_t *lpos;    // [MQ] its position
  float *thr;       // [MQ] score part of lmin (-inf while not full)
  int32_t *flag;    // [MQ] tile may hold an entrant for this query
  uint64_t *lists;  // LDS lists [MQ x k] or nullptr (then lists are in part)
};

__device__ __forceinline__ uint64_t *list_ptr(const TileState &ts, const ScoreArgs &a, int q,
                                              int64_t qg, int64_t S, int64_t s) {
  if (ts.lists) return ts.lists + (int64_t)q * a.k;
  return a.part + (qg * S + s) * a.k;
}

template <int MQ>
__device__ void init_lists(const TileState &ts, const ScoreArgs &a, int64_t qbase, int64_t nu,
                           int64_t S, int64_t s) {
  for (int q = threadIdx.x; q < MQ; q += blockDim.x) {
    ts.lmin[q] = 0ull;
    ts.lpos[q] = 0;
    ts.thr[q] = -__builtin_inff();
    ts.flag[q] = 0;
    int64_t qg = qbase + q;
    if (qg < nu || ts.lists) {
      uint64_t *l = list_ptr(ts, a, q, qg, S, s);
      for (int j = 0; j < a.k; ++j) l[j] = 0ull;
    }
  }
}

// One thread per flagged query scans its dumped tile row.
template <int MQ, int NC, int LD>
__device__ void scan_tile(const TileState &ts, const ScoreArgs &a, const float *dump,
                          int64_t qbase, int64_t nu, int64_t rbase, int64_t S, int64_t s) {
  const int q = threadIdx.x;
  if (q >= MQ) return;
  const int64_t qg = qbase + q;
  if (qg >= nu || !ts.flag[q]) return;
  ts.flag[q] = 0;
  uint64_t *l = list_ptr(ts, a, q, qg, S, s);
  uint64_t mn = ts.lmin[q];
  int mp = ts.lpos[q];
  const float *row = dump + q * LD;
  const int64_t nvalid = a.N - rbase < NC ? a.N - rbase : NC;
  for (int i4 = 0; i4 < NC / 4; ++i4) {
    float4 v = *reinterpret_cast<const float4 *>(row + 4 * i4);
    float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      int i = 4 * i4 + c;
      if (i >= nvalid) break;
      uint64_t key = make_key(vv[c], (uint32_t)(rbase + i));
      if (key > mn) {
        l[mp] = key;
        mn = ~0ull;
        for (int j = 0; j < a.k; ++j) {
          uint64_t x = l[j];
          if (x < mn) {
            mn = x;
            mp = j;
          }
        }
      }
    }
  }
  ts.lmin[q] = mn;
  ts.lpos[q] = mp;
  ts.thr[q] = mn ? unord_score((uint32_t)(mn >> 32)) : -__builtin_inff();
}

template <int MQ>
__device__ void flush_lists(const TileState &ts, const ScoreArgs &a, int64_t qbase, int64_t nu,
                            int64_t S, int64_t s) {
  if (!ts.lists) return;
  const int tot = MQ * a.k;
  for (int t = threadIdx.x; t < tot; t += blockDim.x) {
    int q = t / a.k, j = t - q * a.k;
    int64_t qg = qbase + q;
    if (qg < nu) a.part[(qg * S + s) * a.k + j] = ts.lists[t];
  }
}

// ---------------------------------------------------------------- MFMA path

__device__ __forceinline__ void cvt_fp8x4_to_bf16(uint32_t w, uint32_t &lo, uint32_t &hi) {
  // exact e4m3 -> bf16 (every e4m3 value is representable in bf16)
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  lo = __builtin_bit_cast(uint32_t, a);
  hi = __builtin_bit_cast(uint32_t, b);
}

template <bool FP8>
struct StageRegs {
  uint4 a[FP8 ? 2 : 4];
  uint4 b[4];
};

// Load one K stage of the corpus tile (rows rbase..+NC) and query tile
// (qbase..+MQ) from global memory; out-of-range rows/columns read as zero.
template <bool FP8>
__device__ __forceinline__ void stage_load(StageRegs<FP8> &r, const ScoreArgs &a, int64_t rbase,
                                           int64_t qbase, int64_t nu, int kc) {
  const int tid = threadIdx.x;
  if constexpr (FP8) {
    const uint8_t *C = (const uint8_t *)a.corpus;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int c = tid + kThreads * i;
      int row = c >> 2, c16 = c & 3;
      int64_t gr = rbase + row;
      int col = kc + c16 * 16;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (gr < a.N && col < a.d) v = *reinterpret_cast<const uint4 *>(C + gr * a.d + col);
      r.a[i] = v;
    }
  } else {
    const uint16_t *C = (const uint16_t *)a.corpus;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int c = tid + kThreads * i;
      int row = c >> 3, c8 = c & 7;
      int64_t gr = rbase + row;
      int col = kc + c8 * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (gr < a.N && col < a.d) v = *reinterpret_cast<const uint4 *>(C + gr * a.d + col);
      r.a[i] = v;
    }
  }
  const uint16_t *Q = (const uint16_t *)a.q;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int c = tid + kThreads * i;
    int row = c >> 3, c8 = c & 7;
    int64_t gq = qbase + row;
    int col = kc + c8 * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (gq < nu && col < a.d) v = *reinterpret_cast<const uint4 *>(Q + gq * a.d + col);
    r.b[i] = v;
  }
}

template <bool FP8>
__device__ __forceinline__ void stage_store(const StageRegs<FP8> &r, uint16_t *As, uint16_t *Bs) {
  const int tid = threadIdx.x;
  if constexpr (FP8) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int c = tid + kThreads * i;
      int row = c >> 2, c16 = c & 3;
      uint4 v = r.a[i];
      uint4 o0, o1;
      cvt_fp8x4_to_bf16(v.x, o0.x, o0.y);
      cvt_fp8x4_to_bf16(v.y, o0.z, o0.w);
      cvt_fp8x4_to_bf16(v.z, o1.x, o1.y);
      cvt_fp8x4_to_bf16(v.w, o1.z, o1.w);
      uint16_t *dst = As + row * kLda + c16 * 16;
      *reinterpret_cast<uint4 *>(dst) = o0;
      *reinterpret_cast<uint4 *>(dst + 8) = o1;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int c = tid + kThreads * i;
      int row = c >> 3, c8 = c & 7;
      *reinterpret_cast<uint4 *>(As + row * kLda + c8 * 8) = r.a[i];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int c = tid + kThreads * i;
    int row = c >> 3, c8 = c & 7;
    *reinterpret_cast<uint4 *>(Bs + row * kLda + c8 * 8) = r.b[i];
  }
}

constexpr int kStageBytes = (kNC + kMQ) * kLda * 2;           // one buffer (A + B)
constexpr int kDumpBytes = kMQ * kDumpLd * 4;
constexpr int kMfmaFixed = (2 * kStageBytes > kDumpBytes ? 2 * kStageBytes : kDumpBytes);
constexpr int kSmallBytes = kMQ * (8 + 4 + 4 + 4) + kNC * 4;

__host__ __device__ constexpr int mfma_lds_bytes(bool lds_lists, int k) {
  return kMfmaFixed + kSmallBytes + (lds_lists ? kMQ * k * 8 : 0);
}

// 4 waves as 2 (corpus rows) x 2 (queries); each wave owns a 64 x 64 block of
// scores = 2 x 2 MFMA 32x32 tiles.  MFMA operand A = corpus rows (M), B =
// queries (N), so each lane's accumulators all belong to the same query
// column: one running threshold per lane and query block.
template <bool FP8, bool LDS_LISTS>
__global__ __launch_bounds__(kThreads, 1) void score_partial_mfma(ScoreArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t *stage = reinterpret_cast<uint16_t *>(smem);
  float *dump = reinterpret_cast<float *>(smem);
  unsigned char *p = smem + kMfmaFixed;
  TileState ts;
  ts.lmin = reinterpret_cast<uint64_t *>(p); p += kMQ * 8;
  ts.lpos = reinterpret_cast<int32_t *>(p); p += kMQ * 4;
  ts.thr = reinterpret_cast<float *>(p); p += kMQ * 4;
  ts.flag = reinterpret_cast<int32_t *>(p); p += kMQ * 4;
  float *sscale = reinterpret_cast<float *>(p); p += kNC * 4;
  ts.lists = LDS_LISTS ? reinterpret_cast<uint64_t *>(p) : nullptr;

  const int64_t nu = read_nu(a.n_unique, a.n_unique_dev, a.cap);
  const Split sp = split_for(nu, a.N, kMQ, kNC, a.grid, a.k);
  const int64_t items = sp.qtiles * sp.S;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wr = wv & 1, wq = wv >> 1;
  const int nst = (int)((a.d + kKC - 1) / kKC);

  for (int64_t w = logical_wg(a.grid); w < items; w += a.grid) {
    const int64_t qt = w % sp.qtiles, s = w / sp.qtiles;
    const int64_t t0 = s * sp.ntiles / sp.S, t1 = (s + 1) * sp.ntiles / sp.S;
    const int64_t qbase = qt * kMQ;
    init_lists<kMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
    float tq0 = -__builtin_inff(), tq1 = -__builtin_inff();

    for (int64_t t = t0; t < t1; ++t) {
      const int64_t rbase = t * kNC;
      if (FP8 && tid < kNC) sscale[tid] = (rbase + tid < a.N) ? a.scale[rbase + tid] : 0.0f;
      f32x16 acc[2][2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

      StageRegs<FP8> regs;
      stage_load<FP8>(regs, a, rbase, qbase, nu, 0);
      stage_store<FP8>(regs, stage, stage + kNC * kLda);
      __syncthreads();
      for (int st = 0; st < nst; ++st) {
        uint16_t *As = stage + (st & 1) * (kStageBytes / 2);
        uint16_t *Bs = As + kNC * kLda;
        if (st + 1 < nst) stage_load<FP8>(regs, a, rbase, qbase, nu, (st + 1) * kKC);
        const uint16_t *pa = As + (wr * 64 + (lane & 31)) * kLda + (lane >> 5) * 8;
        const uint16_t *pb = Bs + (wq * 64 + (lane & 31)) * kLda + (lane >> 5) * 8;
#pragma unroll
        for (int kk = 0; kk < kKC; kk += 16) {
          bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(pa + kk);
          bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(pa + 32 * kLda + kk);
          bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(pb + kk);
          bf16x8 b1 = *reinterpret_cast<const bf16x8 *>(pb + 32 * kLda + kk);
          acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
          acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
          acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
          acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
        if (st + 1 < nst) {
          uint16_t *An = stage + ((st + 1) & 1) * (kStageBytes / 2);
          stage_store<FP8>(regs, An, An + kNC * kLda);
        }
        __syncthreads();
      }

      // epilogue: lane owns query column (lane & 31) of each query block and
      // rows 8*(e/4) + 4*(lane/32) + (e%4) of each 32-row block
      const int rsub = 4 * (lane >> 5);
      if (FP8) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float4 sc = *reinterpret_cast<const float4 *>(sscale + wr * 64 + i * 32 + 8 * g + rsub);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              acc[i][j][4 * g + 0] *= sc.x;
              acc[i][j][4 * g + 1] *= sc.y;
              acc[i][j][4 * g + 2] *= sc.z;
              acc[i][j][4 * g + 3] *= sc.w;
            }
          }
      }
      bool hit0 = false, hit1 = false;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          hit0 |= acc[i][0][e] >= tq0;
          hit1 |= acc[i][1][e] >= tq1;
        }
      const int qc0 = wq * 64 + (lane & 31), qc1 = qc0 + 32;
      if (hit0) ts.flag[qc0] = 1;
      if (hit1) ts.flag[qc1] = 1;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r = wr * 64 + i * 32 + 8 * g + rsub;
          float4 v0 = make_float4(acc[i][0][4 * g], acc[i][0][4 * g + 1], acc[i][0][4 * g + 2],
                                  acc[i][0][4 * g + 3]);
          float4 v1 = make_float4(acc[i][1][4 * g], acc[i][1][4 * g + 1], acc[i][1][4 * g + 2],
                                  acc[i][1][4 * g + 3]);
          *reinterpret_cast<float4 *>(dump + qc0 * kDumpLd + r) = v0;
          *reinterpret_cast<float4 *>(dump + qc1 * kDumpLd + r) = v1;
        }
      __syncthreads();
      scan_tile<kMQ, kNC, kDumpLd>(ts, a, dump, qbase, nu, rbase, sp.S, s);
      __syncthreads();
      tq0 = ts.thr[qc0];
      tq1 = ts.thr[qc1];
    }
    flush_lists<kMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- fp32 VALU path

__host__ __device__ constexpr int valu_lds_bytes(bool lds_lists, int k) {
  return (2 * kVNC * kVLd * 4 > kVMQ * kVDumpLd * 4 ? 2 * kVNC * kVLd * 4
                                                    : kVMQ * kVDumpLd * 4) +
         kVMQ * (8 + 4 + 4 + 4) + (lds_lists ? kVMQ * k * 8 : 0);
}

// 16 x 16 threads; thread (ty, tx) computes queries 4*ty.. x rows 4*tx.. .
template <bool LDS_LISTS>
__global__ __launch_bounds__(kThreads) void score_partial_valu(ScoreArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  float *Cs = reinterpret_cast<float *>(smem);       // [kVNC][kVLd]
  float *Qs = Cs + kVNC * kVLd;                       // [kVMQ][kVLd]
  float *dump = reinterpret_cast<float *>(smem);
  constexpr int fixed = (2 * kVNC * kVLd * 4 > kVMQ * kVDumpLd * 4 ? 2 * kVNC * kVLd * 4
                                                                    : kVMQ * kVDumpLd * 4);
  unsigned char *p = smem + fixed;
  TileState ts;
  ts.lmin = reinterpret_cast<uint64_t *>(p); p += kVMQ * 8;
  ts.lpos = reinterpret_cast<int32_t *>(p); p += kVMQ * 4;
  ts.thr = reinterpret_cast<float *>(p); p += kVMQ * 4;
  ts.flag = reinterpret_cast<int32_t *>(p); p += kVMQ * 4;
  ts.lists = LDS_LISTS ? reinterpret_cast<uint64_t *>(p) : nullptr;

  const int64_t nu = read_nu(a.n_unique, a.n_unique_dev, a.cap);
  const Split sp = split_for(nu, a.N, kVMQ, kVNC, a.grid, a.k);
  const int64_t items = sp.qtiles * sp.S;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const float *Q = (const float *)a.q;
  const float *C = (const float *)a.corpus;

  for (int64_t w = logical_wg(a.grid); w < items; w += a.grid) {
    const int64_t qt = w % sp.qtiles, s = w / sp.qtiles;
    const int64_t t0 = s * sp.ntiles / sp.S, t1 = (s + 1) * sp.ntiles / sp.S;
    const int64_t qbase = qt * kVMQ;
    init_lists<kVMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
    for (int64_t t = t0; t < t1; ++t) {
      const int64_t rbase = t * kVNC;
      float acc[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
      for (int64_t kc = 0; kc < a.d; kc += kVKC) {
        for (int e = tid; e < kVNC * kVKC; e += kThreads) {
          int r = e / kVKC, c = e % kVKC;
          int64_t gr = rbase + r, gc = kc + c;
          Cs[r * kVLd + c] = (gr < a.N && gc < a.d) ? C[gr * a.d + gc] : 0.0f;
          int64_t gq = qbase + r;
          Qs[r * kVLd + c] = (gq < nu && gc < a.d) ? Q[gq * a.d + gc] : 0.0f;
        }
        __syncthreads();
        for (int c = 0; c < kVKC; ++c) {
          float qv[4], cv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) qv[i] = Qs[(4 * ty + i) * kVLd + c];
#pragma unroll
          for (int j = 0; j < 4; ++j) cv[j] = Cs[(4 * tx + j) * kVLd + c];
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(qv[i], cv[j], acc[i][j]);
        }
        __syncthreads();
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 4 * ty + i;
        const float th = ts.thr[q];
        bool hit = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) hit |= acc[i][j] >= th;
        if (hit) ts.flag[q] = 1;
        *reinterpret_cast<float4 *>(dump + q * kVDumpLd + 4 * tx) =
            make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
      }
      __syncthreads();
      scan_tile<kVMQ, kVNC, kVDumpLd>(ts, a, dump, qbase, nu, rbase, sp.S, s);
      __syncthreads();
    }
    flush_lists<kVMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- merge

constexpr int kMergeThreads = 1024;

// One workgroup per distinct query: bitonic sort (descending) of its S*k
// slice keys, first k decoded to (score, row).
__global__ __launch_bounds__(kMergeThreads) void topk_merge_kernel(
    const uint64_t *__restrict__ part, int64_t n_unique, const int64_t *__restrict__ n_unique_dev,
    int64_t cap, int64_t N, int k, int mq, int nc, int grid, float *__restrict__ out_s,
    int32_t *__restrict__ out_i) {
  __shared__ uint64_t buf[kMaxSK];
  const int64_t nu = read_nu(n_unique, n_unique_dev, cap);
  const Split sp = split_for(nu, N, mq, nc, grid, k);
  const int tid = threadIdx.x;
  for (int64_t q = blockIdx.x; q < nu; q += gridDim.x) {
    const int n = (int)(sp.S * k);
    int P = 2;
    while (P < n) P <<= 1;
    const uint64_t *src = part + q * sp.S * k;
    for (int i = tid; i < P; i += kMergeThreads) buf[i] = i < n ? src[i] : 0ull;
    __syncthreads();
    for (int size = 2; size <= P; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int t = tid; t < (P >> 1); t += kMergeThreads) {
          int i = 2 * t - (t & (stride - 1));
          int j = i + stride;
          bool desc = (i & size) == 0;
          uint64_t x = buf[i], y = buf[j];
          if ((x < y) == desc) {
            buf[i] = y;
            buf[j] = x;
          }
        }
        __syncthreads();
      }
    }
    for (int j = tid; j < k; j += kMergeThreads) {
      float sc;
      int32_t row;
      decode_key(j < P ? buf[j] : 0ull, sc, row);
      out_s[q * k + j] = sc;
      out_i[q * k + j] = row;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- host side

static int g_grid_cache[64];

int persistent_grid(bool mfma) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (!g_grid_cache[dev]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    int g = cus;  // one persistent workgroup per CU
    g &= ~7;
    if (g < 8) g = 8;
    if (g > kGridMax) g = kGridMax;
    g_grid_cache[dev] = g;
  }
  (void)mfma;
  return g_grid_cache[dev];
}

static size_t partial_bytes(int64_t cap, int64_t N, int mq, int nc, int k) {
  // worst case over n_u in [1, cap] of n_u * S(n_u) * k keys, for any grid
  // size up to kGridMax
  size_t best = 0;
  int64_t qtmax = (cap + mq - 1) / mq;
  for (int64_t qt = 1; qt <= qtmax; ++qt) {
    int64_t nu = qt * mq < cap ? qt * mq : cap;
    Split sp = split_for(nu, N, mq, nc, kGridMax, k);
    size_t b = (size_t)nu * (size_t)sp.S * (size_t)k * 8;
    if (b > best) best = b;
  }
  return (best + 255) & ~(size_t)255;
}

size_t score_workspace_bytes(int64_t cap, int64_t N, int k, int corpus_dtype) {
  if (corpus_dtype == HS_F32) return partial_bytes(cap, N, kVMQ, kVNC, k);
  return partial_bytes(cap, N, kMQ, kNC, k);
}

template <typename K>
static hipError_t launch_with_lds(K kern, int grid, int lds, const ScoreArgs &a, hipStream_t st) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_score_partial(const void *q, const void *corpus, const float *scale, int64_t N,
                                int64_t d, int k, int64_t n_unique, const int64_t *nu_dev,
                                int64_t cap, int corpus_dtype, void *part, hipStream_t st) {
  ScoreArgs a;
  a.q = q;
  a.corpus = corpus;
  a.scale = scale;
  a.N = N;
  a.d = d;
  a.k = k;
  a.n_unique = n_unique;
  a.n_unique_dev = nu_dev;
  a.cap = cap;
  a.part = (uint64_t *)part;
  const bool lds_lists = k <= kListLdsMaxK;
  if (corpus_dtype == HS_F32) {
    a.grid = persistent_grid(false);
    int lds = valu_lds_bytes(lds_lists, k);
    return lds_lists ? launch_with_lds(score_partial_valu<true>, a.grid, lds, a, st)
                     : launch_with_lds(score_partial_valu<false>, a.grid, lds, a, st);
  }
  a.grid = persistent_grid(true);
  int lds = mfma_lds_bytes(lds_lists, k);
  if (corpus_dtype == HS_FP8_E4M3)
    return lds_lists ? launch_with_lds(score_partial_mfma<true, true>, a.grid, lds, a, st)
                     : launch_with_lds(score_partial_mfma<true, false>, a.grid, lds, a, st);
  return lds_lists ? launch_with_lds(score_partial_mfma<false, true>, a.grid, lds, a, st)
                   : launch_with_lds(score_partial_mfma<false, false>, a.grid, lds, a, st);
}

hipError_t launch_topk_merge(const void *part, int64_t n_unique, const int64_t *nu_dev,
                             int64_t cap, int64_t N, int k, int corpus_dtype, float *out_s,
                             int32_t *out_i, hipStream_t st) {
  const bool valu = corpus_dtype == HS_F32;
  const int grid = persistent_grid(!valu);
  int64_t blocks = n_unique >= 0 ? n_unique : cap;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 65535) blocks = 65535;
  hipLaunchKernelGGL(topk_merge_kernel, dim3((unsigned)blocks), dim3(kMergeThreads), 0, st,
                     (const uint64_t *)part, n_unique, nu_dev, cap, N, k, valu ? kVMQ : kMQ,
                     valu ? kVNC : kNC, grid, out_s, out_i);
  return hipGetLastError();
}

}  // namespace hs
