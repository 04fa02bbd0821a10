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
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kMaxSK = 8192;        // bound on S*k (merge list length per query)
constexpr int kListLdsMaxK = 32;    // slice lists live in LDS up to this k
constexpr int kGridMax = 512;       // persistent grid never exceeds this

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
//
// Workgroup = 4 waves (one per SIMD).  Tile = 256 corpus rows x 128 queries;
// wave w owns rows [64w, 64w+64) of the tile for all 128 queries, as 2 x 4
// MFMA 32x32x16 blocks (A = 32 corpus rows, B = 32 queries, fp32 C).  With a
// single wave per SIMD the 32x32x16 form is the one that keeps the matrix
// core busy back to back.
//
// Operand paths, per K chunk of 64:
//   corpus: global -> registers directly (each wave loads only its own rows,
//           so nothing is shared and no LDS is needed), a ring of chunks;
//   queries: global -> registers -> a 3-slot LDS ring, XOR-swizzled by row
//           so that fragment reads are conflict-free.
// Only the query operand is read from LDS: 64 corpus rows reuse each query
// fragment, which keeps LDS traffic near half of its bandwidth at full MFMA
// rate.  Inside an MFMA the K order is free as long as A and B agree, so each
// lane takes the k-slice of a chunk that makes its corpus loads contiguous.
//
// Top-k epilogue, per tile and query: each lane holds 32 scores of each of
// its 4 queries (16 rows of each 32-row block).  It compares their maximum
// with the query's running threshold (registers); only on a hit are single
// scores appended to a small per-query LDS queue, which one thread per query
// then merges into the query's k-list (replace-the-minimum).  A full queue
// leaves the remaining passing scores pending for another round after the
// merge has raised the threshold, so no candidate is lost and none is seen
// twice.  Before the first tile of a work item is filtered, the threshold is
// seeded with the smallest of at least k group maxima of that tile (the 8
// lanes holding a query each split their rows into groups): those maxima are
// k distinct scores, so their minimum never exceeds the true k-th best score.

constexpr int kW2 = 4;                      // waves per workgroup (one per SIMD)
constexpr int kT2 = kW2 * 64;               // threads per workgroup
constexpr int kRB = 2;                      // 32-row blocks per wave
constexpr int kNC2 = kW2 * 32 * kRB;        // 256 rows per tile
constexpr int kKC2 = 64;                    // K per chunk
constexpr int kQcap = 16;                   // queue slots per query
constexpr int kLanesQ = kW2 * 2;            // lanes holding one query in a tile
constexpr int kQB = 4;                      // query blocks of 32 per tile
constexpr int kMQ2 = 32 * kQB;              // 128 queries per tile
constexpr int kVals = 16 * kRB;             // scores per lane and query per tile
constexpr int kRing = 2;                    // corpus chunks held in registers
constexpr int kBP = kMQ2 * 8 / kT2;         // query pieces staged per thread
static_assert(kMQ2 * 8 % kT2 == 0, "query pieces divide evenly");

struct Lds2 {
  uint16_t *bring;   // [3][MQ][64] bf16, swizzled
  uint64_t *queue;   // [MQ][kQcap]
  int32_t *qcount;   // [MQ]
  float *thr0;       // [MQ]
  float *sscale;     // [kNC2]
  int32_t *flags;    // [0] hit epoch, [1] overflow epoch
  float *stash;      // [threads][kVals] scores of one query block (rare path)
  float *gm;         // [MQ][kLanesQ * 8] warm-up group maxima (aliases stash)
  TileState ts;
};

// Warm-up groups per lane and query: the kVals rows a lane holds for one
// query are cut into gpl groups so that kLanesQ * gpl >= k group maxima exist;
// the smallest of them is a valid lower bound for the k-th best score.
// 0 = no warm-up (k too large).
__host__ __device__ constexpr int warm_groups(int k) {
  int g = 1;
  while (g <= 8 && kLanesQ * g < k) g <<= 1;
  return g <= 8 ? g : 0;
}

constexpr int kStashBytes = kT2 * kVals * 4 > kMQ2 * kLanesQ * 8 * 4 ? kT2 * kVals * 4
                                                                      : kMQ2 * kLanesQ * 8 * 4;

__host__ __device__ constexpr int mfma2_lds_bytes(bool lds_lists, int k) {
  return 3 * kMQ2 * kKC2 * 2 + kMQ2 * kQcap * 8 + kMQ2 * 4 + kMQ2 * 4 + kNC2 * 4 + 16 +
         kStashBytes + kMQ2 * (8 + 4 + 4 + 4) + (lds_lists ? kMQ2 * k * 8 : 0);
}

__device__ __forceinline__ void cvt_fp8x4_to_bf16(uint32_t w, uint32_t &lo, uint32_t &hi) {
  // exact e4m3 -> bf16 (every e4m3 value is representable in bf16)
  bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true);
  lo = __builtin_bit_cast(uint32_t, a);
  hi = __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ bf16x8 fp8x8_to_bf16(uint32_t lo, uint32_t hi) {
  uint32_t o0, o1, o2, o3;
  cvt_fp8x4_to_bf16(lo, o0, o1);
  cvt_fp8x4_to_bf16(hi, o2, o3);
  uint4 v = make_uint4(o0, o1, o2, o3);
  return __builtin_bit_cast(bf16x8, v);
}

// 16-byte piece (8 bf16) of a 64-wide K chunk that lane half h feeds to MFMA
// step s.  bf16 corpus rows: the two lane halves load adjacent pieces, so each
// load instruction reads 32 contiguous bytes per row; fp8 rows: each lane
// loads 32 contiguous bytes (4 steps' worth) at once.
template <bool FP8>
__device__ __forceinline__ int kpiece(int h, int s) {
  return FP8 ? 4 * h + s : 2 * s + h;
}

__device__ __forceinline__ int swz(int q, int p) { return q * 64 + ((p ^ (q & 7)) << 3); }

// Per-item state of the top-k epilogue.
struct EpiState {
  int qbase, qvalid, s_;
  int64_t S;
  int epoch;
};

// Row of score j of 32-row block rb held by a lane: 8*(j/4) + 4*h + j%4.
__device__ __forceinline__ int acc_row(int rbase, int rb, int j) {
  return rbase + rb * 32 + 8 * (j >> 2) + (j & 3);
}

// Top-k epilogue of one corpus tile.  `row0` is the corpus row of the tile's
// first loaded row; rows below `rlo` (already scored by the previous tile)
// and at or above N are excluded.
template <bool FP8, bool LDS_LISTS>
__device__ __forceinline__ void tile_epilogue(const Lds2 &L, const ScoreArgs &a,
                                              f32x16 (&acc)[kRB][kQB], float (&thr_r)[kQB],
                                              EpiState &es, int row0, int rlo, bool first) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int N = (int)a.N;
  const float ninf = -__builtin_inff();
  const int rbase = row0 + wv * (32 * kRB) + 4 * h;
  if (FP8) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float4 sc = *reinterpret_cast<const float4 *>(
            L.sscale + wv * (32 * kRB) + rb * 32 + 8 * jj + 4 * h);
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
          acc[rb][qb][4 * jj + 0] *= sc.x;
          acc[rb][qb][4 * jj + 1] *= sc.y;
          acc[rb][qb][4 * jj + 2] *= sc.z;
          acc[rb][qb][4 * jj + 3] *= sc.w;
        }
      }
  }
  // excluded rows never compete: NaN fails every >= test and is ignored by
  // fmaxf
  if (rlo > row0 || row0 + kNC2 > N) {
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int r = acc_row(rbase, rb, j);
        if (r >= N || r < rlo)
#pragma unroll
          for (int qb = 0; qb < kQB; ++qb) acc[rb][qb][j] = __builtin_nanf("");
      }
  }
  const int gpl = warm_groups(a.k);
  if (first && gpl > 0) {
    // warm-up threshold: the smallest of kLanesQ * gpl group maxima
    const int span = kVals / gpl;   // scores per group
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      float *dst = L.gm + (qb * 32 + c) * (kLanesQ * 8) + (wv * 2 + h) * gpl;
      float m = ninf;
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          m = fmaxf(m, acc[rb][qb][j]);
          const int idx = rb * 16 + j;
          if ((idx + 1) % span == 0) {
            dst[idx / span] = m;
            m = ninf;
          }
        }
    }
    __syncthreads();
    if (tid < es.qvalid) {
      const float *v = L.gm + tid * (kLanesQ * 8);
      const int n = kLanesQ * gpl;
      float mn = v[0];
      for (int i = 1; i < n; ++i) mn = fminf(mn, v[i]);
      L.thr0[tid] = mn;
      L.ts.thr[tid] = mn;
    }
    __syncthreads();
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) thr_r[qb] = L.ts.thr[qb * 32 + c];
  }

  // candidate rounds: scores at or above the query threshold go to the
  // query's LDS queue; when a queue is full the remaining bits stay pending
  uint32_t pending[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) pending[qb] = 0;
  float *st = L.stash + tid * kVals;
  for (int round = 0;; ++round) {
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      const int ql = qb * 32 + c;
      const float th = thr_r[qb];
      uint32_t mask = 0;
      if (round == 0) {
        if (ql < es.qvalid) {
          float m = ninf;
#pragma unroll
          for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
            for (int j = 0; j < 16; ++j) m = fmaxf(m, acc[rb][qb][j]);
          if (m >= th) {
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
              for (int j = 0; j < 16; ++j)
                mask |= (acc[rb][qb][j] >= th ? 1u : 0u) << (rb * 16 + j);
          }
        }
      } else {
        mask = pending[qb];
      }
      pending[qb] = 0;
      if (mask) {
        any = true;
        // stash this lane's scores of the block; walk only the passing ones
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            *reinterpret_cast<float4 *>(st + rb * 16 + 4 * jj) =
                make_float4(acc[rb][qb][4 * jj], acc[rb][qb][4 * jj + 1],
                            acc[rb][qb][4 * jj + 2], acc[rb][qb][4 * jj + 3]);
        uint32_t mm = mask;
        while (mm) {
          const int idx = __builtin_ctz(mm);
          const int slot = atomicAdd(&L.qcount[ql], 1);
          if (slot >= kQcap) {
            pending[qb] = mm;
            break;
          }
          L.queue[ql * kQcap + slot] =
              make_key(st[idx], (uint32_t)acc_row(rbase, idx >> 4, idx & 15));
          mm &= mm - 1u;
        }
      }
    }
    if (__ballot(any)) {
      if (lane == 0) L.flags[0] = es.epoch;
    }
    __syncthreads();
    if (L.flags[0] != es.epoch) {
      ++es.epoch;
      break;
    }
    // merge queues into the k-lists, one thread per query
    if (tid < es.qvalid) {
      const int cnt = L.qcount[tid];
      if (cnt > 0) {
        const int n = cnt < kQcap ? cnt : kQcap;
        uint64_t *l = LDS_LISTS ? L.ts.lists + tid * a.k
                                : a.part + ((int64_t)(es.qbase + tid) * es.S + es.s_) * a.k;
        uint64_t mn = L.ts.lmin[tid];
        int mp = L.ts.lpos[tid];
        for (int e = 0; e < n; ++e) {
          const uint64_t key = L.queue[tid * kQcap + e];
          if (key > mn) {
            l[mp] = key;
            mn = ~0ull;
            for (int j2 = 0; j2 < a.k; ++j2) {
              const uint64_t x = l[j2];
              if (x < mn) {
                mn = x;
                mp = j2;
              }
            }
          }
        }
        L.ts.lmin[tid] = mn;
        L.ts.lpos[tid] = mp;
        const float t = mn ? unord_score((uint32_t)(mn >> 32)) : ninf;
        const float t0v = L.thr0[tid];
        L.ts.thr[tid] = t > t0v ? t : t0v;
        L.qcount[tid] = 0;
        if (cnt > kQcap) L.flags[1] = es.epoch;
      }
    }
    __syncthreads();
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) thr_r[qb] = L.ts.thr[qb * 32 + c];
    const bool again = L.flags[1] == es.epoch;
    ++es.epoch;
    if (!again) break;
  }
}

template <bool LDS_LISTS>
__device__ __forceinline__ Lds2 carve_lds(unsigned char *p) {
  Lds2 L;
  L.bring = reinterpret_cast<uint16_t *>(p); p += 3 * kMQ2 * kKC2 * 2;
  L.queue = reinterpret_cast<uint64_t *>(p); p += kMQ2 * kQcap * 8;
  L.qcount = reinterpret_cast<int32_t *>(p); p += kMQ2 * 4;
  L.thr0 = reinterpret_cast<float *>(p); p += kMQ2 * 4;
  L.sscale = reinterpret_cast<float *>(p); p += kNC2 * 4;
  L.flags = reinterpret_cast<int32_t *>(p); p += 16;
  L.stash = reinterpret_cast<float *>(p);
  L.gm = reinterpret_cast<float *>(p); p += kStashBytes;
  L.ts.lmin = reinterpret_cast<uint64_t *>(p); p += kMQ2 * 8;
  L.ts.lpos = reinterpret_cast<int32_t *>(p); p += kMQ2 * 4;
  L.ts.thr = reinterpret_cast<float *>(p); p += kMQ2 * 4;
  L.ts.flag = reinterpret_cast<int32_t *>(p); p += kMQ2 * 4;
  L.ts.lists = LDS_LISTS ? reinterpret_cast<uint64_t *>(p) : nullptr;
  return L;
}

// One K chunk of MFMAs (every query block, including padding ones: a skip
// per block would let the compiler chain MFMAs on one accumulator).
template <bool FP8>
__device__ __forceinline__ void mfma_chunk(f32x16 (&acc)[kRB][kQB], const uint4 (&ab)[kRB][4],
                                           const uint16_t *bs, int c, int h) {
  // all query fragments of the chunk are read up front: with one wave per
  // SIMD nothing else would cover the LDS latency in front of each MFMA
  // group (rows qb*32 + c share (q & 7) with c, so every block's swizzle is
  // block 0's shifted by qb*32 rows)
  bf16x8 bf[4][kQB];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const uint16_t *bsq = bs + swz(c, kpiece<FP8>(h, s));
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
      bf[s][qb] = *reinterpret_cast<const bf16x8 *>(bsq + qb * 32 * kKC2);
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    bf16x8 af[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      if constexpr (FP8) {
        const uint4 v = ab[rb][s >> 1];
        af[rb] = (s & 1) == 0 ? fp8x8_to_bf16(v.x, v.y) : fp8x8_to_bf16(v.z, v.w);
      } else {
        af[rb] = __builtin_bit_cast(bf16x8, ab[rb][s]);
      }
    }
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
        acc[rb][qb] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], bf[s][qb], acc[rb][qb], 0, 0, 0);
  }
  // keep that order through instruction scheduling: LDS reads, then MFMAs
  __builtin_amdgcn_sched_group_barrier(0x100, 4 * kQB, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, 4 * kQB * kRB, 0);
}

// FAST: d is a multiple of 64 * kRing and N >= kNC2.  Then no load ever needs
// a per-lane clamp: every K chunk is whole, the ring turns a whole number of
// times per tile, and the last (ragged) corpus tile is loaded shifted back to
// end at row N, with the rows already scored by the previous tile excluded in
// the epilogue.  Stream positions advance with scalar counters.  Otherwise
// (general d or tiny N) loads clamp per lane and the K walk is padded.
template <bool FP8, bool LDS_LISTS, bool FAST>
__global__ __launch_bounds__(kT2, 1) void score_partial_mfma(ScoreArgs a) {
  static_assert(kT2 == 256, "one wave per SIMD");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const Lds2 L = carve_lds<LDS_LISTS>(smem);

  const int64_t nu = read_nu(a.n_unique, a.n_unique_dev, a.cap);
  const Split sp = split_for(nu, a.N, kMQ2, kNC2, a.grid, a.k);
  const int items = (int)(sp.qtiles * sp.S);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int N = (int)a.N, d = (int)a.d;
  const int nch = (d + kKC2 - 1) / kKC2;
  const float ninf = -__builtin_inff();
  constexpr int esz = FP8 ? 1 : 2;
  constexpr int kAL = FP8 ? 2 : 4;   // 16-byte corpus loads per row block and chunk
  if (tid < 4) L.flags[tid] = 0;
  EpiState es;
  es.epoch = 1;

  // per-lane corpus rows inside a tile and byte columns inside a chunk
  int arow[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) arow[rb] = wv * (32 * kRB) + rb * 32 + c;
  int acol[4];   // element column of load i of a row block
#pragma unroll
  for (int i = 0; i < 4; ++i) acol[i] = FP8 ? 32 * h + 16 * i : 8 * kpiece<false>(h, i);
  // FAST: byte offsets of this lane's corpus pieces from a tile/chunk base
  uint32_t aoff[kRB][4];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) aoff[rb][i] = (uint32_t)(arow[rb] * d + acol[i]) * esz;

  for (int w = logical_wg(a.grid); w < items; w += a.grid) {
    const int qt = w % (int)sp.qtiles;
    es.s_ = w / (int)sp.qtiles;
    es.S = sp.S;
    const int t0 = (int)((int64_t)es.s_ * sp.ntiles / sp.S);
    const int t1 = (int)((int64_t)(es.s_ + 1) * sp.ntiles / sp.S);
    es.qbase = qt * kMQ2;
    es.qvalid = (int)(nu - es.qbase < kMQ2 ? nu - es.qbase : kMQ2);
    const uint16_t *qtile = (const uint16_t *)a.q + (int64_t)es.qbase * d;
    init_lists<kMQ2>(L.ts, a, es.qbase, nu, sp.S, es.s_);
    for (int q = tid; q < kMQ2; q += kT2) {
      L.qcount[q] = 0;
      L.thr0[q] = ninf;
    }
    float thr_r[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) thr_r[qb] = ninf;

    // query pieces this thread stages (global offset always readable; pieces
    // of padding queries repeat the last real query and are never used)
    int brow[kBP], bpc[kBP], bdst[kBP];
    uint32_t bok = 0;
#pragma unroll
    for (int i = 0; i < kBP; ++i) {
      const int piece = tid + kT2 * i;
      const int q = piece >> 3, pp = piece & 7;
      if (q < es.qvalid) bok |= 1u << i;
      brow[i] = (q < es.qvalid ? q : es.qvalid - 1) * d;
      bpc[i] = 8 * pp;
      bdst[i] = swz(q, pp);
    }

    const int nchp = FAST ? nch : (nch + kRing - 1) / kRing * kRing;
    const int ntl = t1 - t0;
    const int total = ntl * nchp;
    uint4 abuf[kRing][kRB][4];
    uint4 bst[2][kBP];   // query chunks in flight: loaded one step before stored
    // first corpus row loaded for a tile (FAST shifts the ragged last tile)
    auto tile_row0 = [&](int tile) {
      int r0 = tile * kNC2;
      if (FAST && r0 > N - kNC2) r0 = N - kNC2;
      return r0;
    };
    // stream positions (FAST): next corpus chunk to load, next query chunk
    int a_tl = 0, a_kc = 0, b_kc = 0, b_slot = 0, r_slot = 0;
    static_assert(kRing % 2 == 0, "query staging parity follows the ring");
    auto load_a = [&](int g, uint4 (&dst)[kRB][4]) {
      if constexpr (FAST) {
        const int tl = a_tl < ntl ? a_tl : ntl - 1;
        const unsigned char *base = (const unsigned char *)a.corpus +
                                    ((int64_t)tile_row0(t0 + tl) * d + a_kc * kKC2) * esz;
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
          for (int i = 0; i < kAL; ++i)
            dst[rb][i] = *reinterpret_cast<const uint4 *>(base + aoff[rb][i]);
        if (++a_kc == nch) {
          a_kc = 0;
          ++a_tl;
        }
      } else {
        if (g > total - 1) g = total - 1;
        const int tile = t0 + g / nchp;
        int kc = (g % nchp) * kKC2;
        if (kc > (nch - 1) * kKC2) kc = (nch - 1) * kKC2;   // padding chunk: any data
        const int rmax = N - 1 - tile * kNC2;          // last valid row in tile
        const int cmax = d - (FP8 ? 16 : 8) - kc;      // last valid piece column
        const unsigned char *base = (const unsigned char *)a.corpus +
                                    ((int64_t)tile * kNC2 * d + kc) * esz;
#pragma unroll
        for (int rb = 0; rb < kRB; ++rb) {
          const int r = arow[rb] < rmax ? arow[rb] : rmax;
#pragma unroll
          for (int i = 0; i < kAL; ++i) {
            const int cc = acol[i] < cmax ? acol[i] : cmax;
            dst[rb][i] = *reinterpret_cast<const uint4 *>(base + (uint32_t)(r * d + cc) * esz);
          }
        }
      }
    };
    auto load_b = [&](int g, uint4 (&bs)[kBP]) {
      int kc;
      if constexpr (FAST) {
        kc = b_kc * kKC2;
        if (++b_kc == nch) b_kc = 0;
      } else {
        kc = (g % nchp) * kKC2;
        if (kc > (nch - 1) * kKC2) kc = (nch - 1) * kKC2;
      }
      const uint16_t *base = qtile + kc;
#pragma unroll
      for (int i = 0; i < kBP; ++i) {
        int col = bpc[i];
        if (!FAST && kc + col > d - 8) col = d - 8 - kc;
        bs[i] = *reinterpret_cast<const uint4 *>(base + brow[i] + col);
      }
    };
    auto store_b = [&](int g, const uint4 (&bs)[kBP]) {
      int slot, kc;
      if constexpr (FAST) {
        slot = b_slot;
        if (++b_slot == 3) b_slot = 0;
        kc = 0;
      } else {
        slot = g % 3;
        kc = (g % nchp) * kKC2;
      }
      uint16_t *base = L.bring + slot * (kMQ2 * kKC2);
#pragma unroll
      for (int i = 0; i < kBP; ++i) {
        uint4 v = bs[i];
        if (!FAST) {
          const bool ok = ((bok >> i) & 1u) && kc + bpc[i] < d;
          v.x = ok ? v.x : 0u;
          v.y = ok ? v.y : 0u;
          v.z = ok ? v.z : 0u;
          v.w = ok ? v.w : 0u;
        }
        *reinterpret_cast<uint4 *>(base + bdst[i]) = v;
      }
    };
    if (total > 0) {
      load_b(0, bst[0]);
      store_b(0, bst[0]);
      load_b(1, bst[1]);
      store_b(1, bst[1]);
      load_b(2, bst[0]);
#pragma unroll
      for (int r = 0; r < kRing - 1; ++r) load_a(r, abuf[r]);
    }
    __syncthreads();

    f32x16 acc[kRB][kQB];
    for (int tl = 0; tl < ntl; ++tl) {
      const int tile = t0 + tl;
      const int row0 = tile_row0(tile);
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[rb][qb][e] = 0.0f;
      if (FP8) {
        for (int t = tid; t < kNC2; t += kT2) {
          const int r = row0 + t;
          L.sscale[t] = r < N ? a.scale[r] : 0.0f;
        }
      }
      for (int kc4 = 0; kc4 < nchp; kc4 += kRing) {
#pragma unroll
        for (int r = 0; r < kRing; ++r) {
          const int g = tl * nchp + kc4 + r;
          // query chunk g+2 was loaded a full step ago; its LDS slot was last
          // read in step g-1 (behind the previous barrier).  Then issue, in
          // this order for the in-order vmcnt waits, the query chunk g+3 and
          // the corpus chunk g+kRing-1.
          store_b(g + 2, bst[r & 1]);
          load_b(g + 3, bst[(r + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
          load_a(g + kRing - 1, abuf[(r + kRing - 1) % kRing]);
          __builtin_amdgcn_sched_barrier(0);
          int slot;
          if constexpr (FAST) {
            slot = r_slot;
            if (++r_slot == 3) r_slot = 0;
          } else {
            slot = g % 3;
          }
          mfma_chunk<FP8>(acc, abuf[r], L.bring + slot * (kMQ2 * kKC2), c, h);
          __syncthreads();
        }
      }
      tile_epilogue<FP8, LDS_LISTS>(L, a, acc, thr_r, es, row0, tile * kNC2, tl == 0);
    }
    flush_lists<kMQ2>(L.ts, a, es.qbase, nu, sp.S, es.s_);
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
  return partial_bytes(cap, N, kMQ2, kNC2, k);
}

template <typename K>
static hipError_t launch_with_lds(K kern, int grid, int threads, int lds, const ScoreArgs &a,
                                  hipStream_t st) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(threads), lds, st, a);
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
    return lds_lists ? launch_with_lds(score_partial_valu<true>, a.grid, kThreads, lds, a, st)
                     : launch_with_lds(score_partial_valu<false>, a.grid, kThreads, lds, a, st);
  }
  a.grid = persistent_grid(true);
  int lds = mfma2_lds_bytes(lds_lists, k);
  const bool fast = d % (kKC2 * kRing) == 0 && N >= kNC2;
#define HS_LAUNCH(F8, LL, FA) \
  return launch_with_lds(score_partial_mfma<F8, LL, FA>, a.grid, kT2, lds, a, st)
  if (corpus_dtype == HS_FP8_E4M3) {
    if (lds_lists) { if (fast) HS_LAUNCH(true, true, true); HS_LAUNCH(true, true, false); }
    if (fast) HS_LAUNCH(true, false, true);
    HS_LAUNCH(true, false, false);
  }
  if (lds_lists) { if (fast) HS_LAUNCH(false, true, true); HS_LAUNCH(false, true, false); }
  if (fast) HS_LAUNCH(false, false, true);
  HS_LAUNCH(false, false, false);
#undef HS_LAUNCH
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
                     (const uint64_t *)part, n_unique, nu_dev, cap, N, k, valu ? kVMQ : kMQ2,
                     valu ? kVNC : kNC2, grid, out_s, out_i);
  return hipGetLastError();
}

}  // namespace hs
