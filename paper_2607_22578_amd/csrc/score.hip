// Steps 3 and 4 for fp32 inputs, the cross-slice merge of step 4, and the
// host-side dispatch of the scoring kernels.
//
// HeraSys runs one retrieval per fused node (Sec. 3.3 (I)) and batches ready
// nodes of the same type (Appendix A, batching constraint); a retrieval node's
// result is its Top-K chunks (Eq. 2 parameters; Sec. 4.1 workloads).  Here the
// batch is the n_u distinct queries and the retrieval is exact inner product.
//
// Phase 1 (score_partial_*): one persistent kernel.  Work items are (query
// tile, corpus slice) pairs (make_split), so the grid is filled whatever n_u
// turns out to be.  bf16 and fp8 corpora run on the matrix cores
// (score_mfma.hip); fp32 inputs run score_partial_valu below: plain VALU FMA
// tiles through LDS, then each query with a possible entrant has its tile row
// merged into the query's k best (score, row) keys of this slice: by one
// wave that ranks the tile's keys and the list's together (k <= 32: the list
// lives in LDS and stays sorted), else by one thread that replaces the list's
// minimum key by key.
// Phase 2 (topk_merge_kernel): per query, the S slice lists (S*k keys) are
// filtered (empty keys, and keys below the query's shared threshold on the
// matrix-core path), the rest sorted and the first k written out.
//
// Result keys order by (score desc, row asc), so ties always go to the lower
// corpus row, independently of which slice or lane saw them.
#include "common.h"

namespace hs {

constexpr int kThreads = 256;
constexpr int kMaxSK = 8192;        // bound on S*k (merge list length per query)
constexpr int kListLdsMaxK = 32;    // slice lists live in LDS up to this k (fp32 path)
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
  int64_t smax = kMaxSK / k;
  return make_split(nu, N, mq, nc, grid, smax < 1 ? 1 : smax);
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

// LDS lists (k <= kListLdsMaxK): one wave per flagged query.  Lane i holds
// the key of tile row i (0 past the corpus end); every key of the union of
// those NC keys and the query's k list keys is ranked by counting the larger
// ones (keys are distinct, except the empty key 0), and the nonzero keys
// ranked below k are written to their rank.  The list thus stays sorted in
// descending order, positions past its nonzero keys keep 0, and the key of
// rank k-1 is its new minimum.  u is this wave's [NC + kListLdsMaxK] scratch.
template <int MQ, int NC, int LD>
__device__ void scan_tile_wave(const TileState &ts, const ScoreArgs &a, const float *dump,
                               uint64_t *u, int64_t qbase, int64_t nu, int64_t rbase) {
  static_assert(NC == kWave, "one tile row per lane");
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int nw = blockDim.x / kWave;
  const int k = a.k;
  const int64_t nvalid = a.N - rbase < NC ? a.N - rbase : NC;
  for (int q = wave; q < MQ; q += nw) {
    if (qbase + q >= nu || !ts.flag[q]) continue;
    uint64_t *l = ts.lists + (int64_t)q * k;
    const uint64_t x0 = lane < nvalid ? make_key(dump[q * LD + lane], (uint32_t)(rbase + lane))
                                      : 0ull;
    const uint64_t x1 = lane < k ? l[lane] : 0ull;
    u[lane] = x0;
    if (lane < kListLdsMaxK) u[NC + lane] = x1;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int r0 = 0, r1 = 0;
    for (int j = 0; j < NC + kListLdsMaxK; j += 8) {
      uint64_t b[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) b[t] = u[j + t];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        r0 += b[t] > x0 ? 1 : 0;
        r1 += b[t] > x1 ? 1 : 0;
      }
    }
    if (x0 != 0ull && r0 < k) l[r0] = x0;
    if (x1 != 0ull && r1 < k) l[r1] = x1;
    if (x0 != 0ull && r0 == k - 1) {
      ts.lmin[q] = x0;
      ts.thr[q] = unord_score((uint32_t)(x0 >> 32));
    }
    if (x1 != 0ull && r1 == k - 1) {
      ts.lmin[q] = x1;
      ts.thr[q] = unord_score((uint32_t)(x1 >> 32));
    }
    if (lane == 0) ts.flag[q] = 0;
    // the scratch is rewritten for the next query only after every lane
    // has read it
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
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

// ---------------------------------------------------------------- fp32 VALU path

__host__ __device__ constexpr int valu_lds_bytes(bool lds_lists, int k) {
  return (2 * kVNC * kVLd * 4 > kVMQ * kVDumpLd * 4 ? 2 * kVNC * kVLd * 4
                                                    : kVMQ * kVDumpLd * 4) +
         kVMQ * (8 + 4 + 4 + 4) +
         (lds_lists ? kVMQ * k * 8 + kThreads / kWave * (kVNC + kListLdsMaxK) * 8 : 0);
}

constexpr int kVLoads = kVNC * kVKC / kThreads;   // corpus (and query) floats per thread
static_assert(kVNC == kVMQ && kVLoads * kThreads == kVNC * kVKC, "chunk split");

// A thread's share of K chunk kc: corpus rows rbase + r and query rows
// qbase + r, columns kc + c, 0 past the corpus, the live queries or d.
__device__ __forceinline__ void valu_fetch(float (&cr)[kVLoads], float (&qr)[kVLoads],
                                           const float *C, const float *Q, const ScoreArgs &a,
                                           int64_t rbase, int64_t qbase, int64_t nu, int64_t kc,
                                           int tid) {
#pragma unroll
  for (int u = 0; u < kVLoads; ++u) {
    const int e = tid + u * kThreads, r = e / kVKC, c = e % kVKC;
    const int64_t gr = rbase + r, gc = kc + c, gq = qbase + r;
    cr[u] = (gr < a.N && gc < a.d) ? C[gr * a.d + gc] : 0.0f;
    qr[u] = (gq < nu && gc < a.d) ? Q[gq * a.d + gc] : 0.0f;
  }
}

// One K chunk of a thread's register tile: NI of its queries (ty + 16 i,
// i < NI) by its four rows 4 tx + j.
template <int NI>
__device__ __forceinline__ void valu_chunk(float (&acc)[4][4], const float *Qs, const float *Cs,
                                           int ty, int tx) {
  for (int c = 0; c < kVKC; ++c) {
    float qv[NI], cv[4];
#pragma unroll
    for (int i = 0; i < NI; ++i) qv[i] = Qs[(ty + 16 * i) * kVLd + c];
#pragma unroll
    for (int j = 0; j < 4; ++j) cv[j] = Cs[(4 * tx + j) * kVLd + c];
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(qv[i], cv[j], acc[i][j]);
  }
}

// Registers of valu_fetch into the LDS chunk.
__device__ __forceinline__ void valu_stage(const float (&cr)[kVLoads], const float (&qr)[kVLoads],
                                           float *Cs, float *Qs, int tid) {
#pragma unroll
  for (int u = 0; u < kVLoads; ++u) {
    const int e = tid + u * kThreads, r = e / kVKC, c = e % kVKC;
    Cs[r * kVLd + c] = cr[u];
    Qs[r * kVLd + c] = qr[u];
  }
}

__device__ __forceinline__ void valu_multiply(int ni, float (&acc)[4][4], const float *Qs,
                                              const float *Cs, int ty, int tx) {
  switch (ni) {
    case 4: valu_chunk<4>(acc, Qs, Cs, ty, tx); break;
    case 3: valu_chunk<3>(acc, Qs, Cs, ty, tx); break;
    case 2: valu_chunk<2>(acc, Qs, Cs, ty, tx); break;
    case 1: valu_chunk<1>(acc, Qs, Cs, ty, tx); break;
    default: break;
  }
}

// 16 x 16 threads; thread (ty, tx) computes queries ty + 16 i (i < 4) x rows
// 4 tx + j (j < 4).  Queries are interleaved over the waves (wave w holds
// ty = 4w .. 4w+3), so a tile with few live queries spreads them over all
// four SIMDs, and each wave multiplies only the query rows i that are live
// for one of its lanes (a wave-uniform count).
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
  uint64_t *wave_u = LDS_LISTS ? reinterpret_cast<uint64_t *>(p) + kVMQ * a.k +
                                     (threadIdx.x / kWave) * (kVNC + kListLdsMaxK)
                               : nullptr;

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
    const int64_t live = nu - qbase;   // >= 1
    const int lo = 4 * (tid >> 6);     // smallest ty of this wave
    const int ni = live <= lo ? 0 : (live - lo + 15) / 16 > 4 ? 4 : (int)((live - lo + 15) / 16);
    init_lists<kVMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
    for (int64_t t = t0; t < t1; ++t) {
      const int64_t rbase = t * kVNC;
      float acc[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
      // K chunks are loaded into registers two ahead of the one being
      // multiplied (two register sets in turn), so their memory latency
      // overlaps the FMAs and the loads of the next chunk
      float cr0[kVLoads], qr0[kVLoads], cr1[kVLoads], qr1[kVLoads];
      valu_fetch(cr0, qr0, C, Q, a, rbase, qbase, nu, 0, tid);
      if (kVKC < a.d) valu_fetch(cr1, qr1, C, Q, a, rbase, qbase, nu, kVKC, tid);
      for (int64_t kc = 0; kc < a.d; kc += 2 * kVKC) {
        valu_stage(cr0, qr0, Cs, Qs, tid);
        __syncthreads();
        if (kc + 2 * kVKC < a.d) valu_fetch(cr0, qr0, C, Q, a, rbase, qbase, nu, kc + 2 * kVKC, tid);
        valu_multiply(ni, acc, Qs, Cs, ty, tx);
        __syncthreads();
        if (kc + kVKC >= a.d) break;
        valu_stage(cr1, qr1, Cs, Qs, tid);
        __syncthreads();
        if (kc + 3 * kVKC < a.d) valu_fetch(cr1, qr1, C, Q, a, rbase, qbase, nu, kc + 3 * kVKC, tid);
        valu_multiply(ni, acc, Qs, Cs, ty, tx);
        __syncthreads();
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = ty + 16 * i;
        const float th = ts.thr[q];
        bool hit = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) hit |= acc[i][j] >= th;
        if (hit) ts.flag[q] = 1;
        *reinterpret_cast<float4 *>(dump + q * kVDumpLd + 4 * tx) =
            make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
      }
      __syncthreads();
      if (LDS_LISTS)
        scan_tile_wave<kVMQ, kVNC, kVDumpLd>(ts, a, dump, wave_u, qbase, nu, rbase);
      else
        scan_tile<kVMQ, kVNC, kVDumpLd>(ts, a, dump, qbase, nu, rbase, sp.S, s);
      __syncthreads();
    }
    flush_lists<kVMQ>(ts, a, qbase, nu, sp.S, s);
    __syncthreads();
  }
}

// ---------------------------------------------------------------- merge

constexpr int kMergeThreads = 1024;
constexpr int kMergeRankMax = 2048;   // survivors ranked by counting up to this many

// One workgroup per distinct query.  Its S*k slice keys are compacted into
// LDS, dropping empty keys, keys below the k-th largest list head when the
// lists are sorted, and, when a shared threshold is given, keys whose score
// is below it (each a lower bound of the query's k-th best, so every key of
// the final k survives); the survivors are sorted (bitonic,
// descending; up to kMergeRankMax survivors are ranked by counting the
// survivors above each instead) and the first k decoded to (score, row),
// ranks past the survivors padded with (-inf, -1).
__global__ __launch_bounds__(kMergeThreads) void topk_merge_kernel(
    const uint64_t *__restrict__ part, const uint32_t *__restrict__ thr, int64_t n_unique,
    const int64_t *__restrict__ n_unique_dev, int64_t cap, int64_t N, int k, int mq, int nc,
    int64_t smax, int grid, int sorted, float *__restrict__ out_s, int32_t *__restrict__ out_i) {
  __shared__ uint64_t buf[kMaxSK + 8];
  __shared__ uint64_t heads[kMergeThreads];
  __shared__ uint64_t head_cut;
  __shared__ int count;
  const int64_t nu = read_nu(n_unique, n_unique_dev, cap);
  const Split sp = make_split(nu, N, mq, nc, grid, smax);
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int n = (int)(sp.S * k);
  for (int64_t q = blockIdx.x; q < nu; q += gridDim.x) {
    const uint32_t t = thr ? thr[q] : 0u;
    const uint64_t *src = part + q * sp.S * k;
    if (tid == 0) {
      count = 0;
      head_cut = 0ull;
    }
    // With lists sorted in descending order, the k-th largest of the S list
    // heads is also a lower bound of the query's k-th best key: the heads
    // are keys of distinct rows (empty heads are 0 and tie, leaving the cut
    // at 0 when fewer than k slices kept anything).
    const bool use_heads = sorted && sp.S >= k && sp.S <= kMergeThreads;
    if (use_heads && tid < sp.S) heads[tid] = src[(int64_t)tid * k];
    __syncthreads();
    if (use_heads && tid < sp.S) {
      const uint64_t hk = heads[tid];
      int r = 0;
      for (int j = 0; j < (int)sp.S; ++j) r += heads[j] > hk ? 1 : 0;
      if (r == k - 1 && hk != 0ull) head_cut = hk;
    }
    __syncthreads();
    const uint64_t cut = head_cut;
    for (int i0 = 0; i0 < n; i0 += kMergeThreads) {
      const int i = i0 + tid;
      const uint64_t key = i < n ? src[i] : 0ull;
      const bool keep = key != 0ull && (uint32_t)(key >> 32) >= t && key >= cut;
      const uint64_t mask = __builtin_amdgcn_ballot_w64(keep);
      int base = 0;
      if (lane == 0 && mask) base = atomicAdd(&count, __popcll(mask));
      base = __shfl(base, 0);
      if (keep) buf[base + __popcll(mask & ((1ull << lane) - 1ull))] = key;
    }
    __syncthreads();
    const int m = count;
    if (m <= kMergeRankMax) {
      // rank = number of survivors above (keys are distinct: one per row);
      // the survivors are padded with empty keys to a multiple of 8 so that
      // eight independent reads are in flight at a time
      const int m8 = (m + 7) & ~7;
      for (int i = m + tid; i < m8; i += kMergeThreads) buf[i] = 0ull;
      __syncthreads();
      for (int u = tid; u < m; u += kMergeThreads) {
        const uint64_t key = buf[u];
        int r = 0;
        for (int j = 0; j < m8; j += 8) {
          uint64_t b[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) b[t] = buf[j + t];
#pragma unroll
          for (int t = 0; t < 8; ++t) r += b[t] > key ? 1 : 0;
        }
        if (r < k) {
          float sc;
          int32_t row;
          decode_key(key, sc, row);
          out_s[q * k + r] = sc;
          out_i[q * k + r] = row;
        }
      }
      for (int j = m + tid; j < k; j += kMergeThreads) {
        out_s[q * k + j] = -__builtin_inff();
        out_i[q * k + j] = -1;
      }
    } else {
      int P = 2;
      while (P < m) P <<= 1;
      for (int i = m + tid; i < P; i += kMergeThreads) buf[i] = 0ull;
      __syncthreads();
      for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
          for (int u = tid; u < (P >> 1); u += kMergeThreads) {
            const int i = 2 * u - (u & (stride - 1));
            const int j = i + stride;
            const bool desc = (i & size) == 0;
            const uint64_t x = buf[i], y = buf[j];
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
        decode_key(j < m ? buf[j] : 0ull, sc, row);
        out_s[q * k + j] = sc;
        out_i[q * k + j] = row;
      }
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

size_t mfma_partial_bytes(int64_t cap, int64_t N, int k, int grid_max);
size_t mfma_qtile_offset(int64_t cap, int64_t N, int k, int grid_max);
size_t mfma_qtile_bytes(int64_t cap, int64_t d);
size_t mfma_part_offset(int64_t cap, int64_t N, int k, int grid_max);
void mfma_split_params(int *mq, int *nc, int64_t *smax, int k);
hipError_t launch_score_mfma(const void *q, const void *corpus, const float *scale, int64_t N,
                             int64_t d, int k, int64_t n_unique, const int64_t *nu_dev,
                             int64_t cap, bool fp8, bool tiled, void *ws, hipStream_t st);

static size_t partial_bytes(int64_t cap, int64_t N, int mq, int nc, int k) {
  // worst case over n_u in [1, cap] of n_u * S(n_u) * k keys, for any grid
  // size up to kGridMax
  size_t best = 0;
  int64_t qtmax = (cap + mq - 1) / mq;
  for (int64_t qt = 1; qt <= qtmax; ++qt) {
    int64_t nu = qt * mq < cap ? qt * mq : cap;
    for (int g = 8; g <= kGridMax; g += 8) {
      Split sp = split_for(nu, N, mq, nc, g, k);
      size_t b = (size_t)nu * (size_t)sp.S * (size_t)k * 8;
      if (b > best) best = b;
    }
  }
  return (best + 255) & ~(size_t)255;
}

size_t score_workspace_bytes(int64_t cap, int64_t N, int64_t d, int k, int corpus_dtype) {
  if (corpus_dtype == HS_F32) return partial_bytes(cap, N, kVMQ, kVNC, k);
  return mfma_qtile_offset(cap, N, k, kGridMax) + mfma_qtile_bytes(cap, d);
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
                                int64_t cap, int corpus_dtype, bool tiled, void *part,
                                hipStream_t st) {
  if (corpus_dtype != HS_F32)
    return launch_score_mfma(q, corpus, scale, N, d, k, n_unique, nu_dev, cap,
                             corpus_dtype == HS_FP8_E4M3, tiled, part, st);
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
  a.grid = persistent_grid(false);
  int lds = valu_lds_bytes(lds_lists, k);
  return lds_lists ? launch_with_lds(score_partial_valu<true>, a.grid, kThreads, lds, a, st)
                   : launch_with_lds(score_partial_valu<false>, a.grid, kThreads, lds, a, st);
}

hipError_t launch_topk_merge(const void *part, int64_t n_unique, const int64_t *nu_dev,
                             int64_t cap, int64_t N, int k, int corpus_dtype, float *out_s,
                             int32_t *out_i, hipStream_t st) {
  const bool valu = corpus_dtype == HS_F32;
  const int grid = persistent_grid(!valu);
  int64_t blocks = n_unique >= 0 ? n_unique : cap;
  if (blocks <= 0) return hipSuccess;
  if (blocks > 65535) blocks = 65535;
  int mq = kVMQ, nc = kVNC;
  int64_t smax = kMaxSK / k;
  if (smax < 1) smax = 1;
  const uint32_t *thr = nullptr;
  if (!valu) {
    mfma_split_params(&mq, &nc, &smax, k);
    // the matrix-core path starts its workspace with the shared thresholds
    // and keeps its partial lists after its other scratch
    thr = (const uint32_t *)part;
    part = (const unsigned char *)part + mfma_part_offset(cap, N, k, kGridMax);
  }
  // a persistent grid of at most two workgroups per CU loops over queries
  if (blocks > 2 * (int64_t)grid) blocks = 2 * (int64_t)grid;
  hipLaunchKernelGGL(topk_merge_kernel, dim3((unsigned)blocks), dim3(kMergeThreads), 0, st,
                     (const uint64_t *)part, thr, n_unique, nu_dev, cap, N, k, mq, nc, smax, grid,
                     valu && k > kListLdsMaxK ? 0 : 1, out_s, out_i);
  return hipGetLastError();
}

}  // namespace hs
