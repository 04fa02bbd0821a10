// Step 1: signature matching -- group R request keys.
//
// HeraSys Sec. 3.3 (I): a node whose signature matches a node already in the
// window is fused into it; Eq. (3) aggregates over the merged set M(v*).  The
// paper detects matches with a hash map (Appendix B.3, Phase 1).  On the GPU
// the same groups come out of a stable sort of (key, request) pairs, which
// also makes every output canonical: distinct keys ascending, the survivor of
// a group is its earliest request, counts[g] = |M(v*)|, inverse[i] = group.
//
// Three paths:
//   R <= kHashMax  : one workgroup groups the keys in an LDS hash table
//                    (first request by atomic min, group size by atomic add),
//                    orders the distinct keys by counting, for each, the
//                    distinct keys below it, and maps every request to its
//                    group through the table;
//   R <= kSmallMax : one workgroup sorts (key, idx) in LDS with a bitonic
//                    network and compacts in the same launch;
//   larger R       : LSD radix sort, 8-bit digits over (key - min) so only
//                    the bits that vary are sorted (the pass count is read on
//                    the device; surplus passes exit at once), stable local
//                    ranking with wavefront ballots, then head flags, a
//                    block-prefix compaction and a counts pass.
#include "common.h"

namespace hs {

constexpr int kSmallMax = 4096;
constexpr int kSmallThreads = 1024;
constexpr int kRadixThreads = 256;
constexpr int kRadixItems = 16;
constexpr int kTile = kRadixThreads * kRadixItems;  // keys per block
constexpr int kRadixBits = 8;
constexpr int kBins = 1 << kRadixBits;

__device__ __forceinline__ uint64_t map_key(int64_t k) {
  return (uint64_t)k ^ 0x8000000000000000ull;
}
__device__ __forceinline__ int64_t unmap_key(uint64_t u) {
  return (int64_t)(u ^ 0x8000000000000000ull);
}

// Inclusive prefix sum over a block; returns the inclusive value for this
// thread and the block total.  `wsum` needs blockDim/64 + 1 entries.
template <int NT>
__device__ __forceinline__ uint32_t block_inclusive_scan(uint32_t v, uint32_t *wsum,
                                                         uint32_t &total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int i = 0; i < NT / 64; ++i) {
      uint32_t t = wsum[i];
      wsum[i] = acc;
      acc += t;
    }
    wsum[NT / 64] = acc;
  }
  __syncthreads();
  total = wsum[NT / 64];
  uint32_t r = x + wsum[w];
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------- small R

__global__ __launch_bounds__(kSmallThreads) void dedup_small_kernel(
    const int64_t *__restrict__ keys, int R, int P, int64_t *__restrict__ uk,
    int32_t *__restrict__ fi, int32_t *__restrict__ cnt, int32_t *__restrict__ inv,
    int64_t *__restrict__ nu_out) {
  __shared__ uint64_t sk[kSmallMax];
  __shared__ int32_t si[kSmallMax];
  __shared__ uint32_t wsum[kSmallThreads / 64 + 1];
  const int tid = threadIdx.x;
  for (int p = tid; p < P; p += kSmallThreads) {
    if (p < R) {
      sk[p] = map_key(keys[p]);
      si[p] = p;
    } else {  // padding sorts after every real (key, idx) pair
      sk[p] = ~0ull;
      si[p] = 0x7FFFFFFF;
    }
  }
  __syncthreads();
  // bitonic sort of (key, idx) ascending
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < (P >> 1); t += kSmallThreads) {
        int i = 2 * t - (t & (stride - 1));
        int j = i + stride;
        bool up = (i & size) == 0;
        uint64_t ki = sk[i], kj = sk[j];
        int32_t ii = si[i], ij = si[j];
        bool gt = ki > kj || (ki == kj && ii > ij);
        if (gt == up) {
          sk[i] = kj; sk[j] = ki;
          si[i] = ij; si[j] = ii;
        }
      }
      __syncthreads();
    }
  }
  // heads and group ids: thread t owns positions [t*E, t*E + E)
  constexpr int E = kSmallMax / kSmallThreads;
  int64_t myk[E];
  int32_t myi[E];
  bool head[E];
  uint32_t h = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    int p = tid * E + e;
    myk[e] = 0;
    myi[e] = 0;
    head[e] = false;
    if (p < R) {
      myk[e] = unmap_key(sk[p]);
      myi[e] = si[p];
      head[e] = (p == 0) || (sk[p] != sk[p - 1]);
      h += head[e];
    }
  }
  uint32_t total;
  uint32_t incl = block_inclusive_scan<kSmallThreads>(h, wsum, total);
  uint32_t g = incl - h;  // heads before this thread
  // si is free now: reuse it for group start positions
#pragma unroll
  for (int e = 0; e < E; ++e) {
    int p = tid * E + e;
    if (p < R) {
      if (head[e]) {
        uk[g] = myk[e];
        fi[g] = myi[e];
        si[g] = p;
        ++g;
      }
      inv[myi[e]] = (int32_t)(g - 1);
    }
  }
  __syncthreads();
  if (cnt) {
    for (int q = tid; q < (int)total; q += kSmallThreads) {
      int end = (q + 1 < (int)total) ? si[q + 1] : R;
      cnt[q] = end - si[q];
    }
  }
  if (tid == 0) *nu_out = (int64_t)total;
}

// ---------------------------------------------------------------- hash path

constexpr int kHashMax = 2048;
constexpr int kHashSlots = 2 * kHashMax;   // load factor at most 1/2
constexpr int kHashPer = kHashMax / kSmallThreads;

__global__ __launch_bounds__(kSmallThreads) void dedup_hash_kernel(
    const int64_t *__restrict__ keys, int R, int64_t *__restrict__ uk, int32_t *__restrict__ fi,
    int32_t *__restrict__ cnt, int32_t *__restrict__ inv, int64_t *__restrict__ nu_out) {
  // Mapped keys (map_key: order-preserving to unsigned) in open addressing
  // with linear probing; mapped value 0 marks an empty slot, so the one key
  // that maps to 0 (INT64_MIN) is counted in a group of its own (zmin, zcnt).
  __shared__ unsigned long long hk[kHashSlots];
  __shared__ int32_t hmin[kHashSlots];   // first request; later the group id
  __shared__ int32_t hcnt[kHashSlots];
  __shared__ unsigned long long ck[kHashMax + 8];   // distinct mapped keys
  __shared__ int32_t cslot[kHashMax + 1];           // their slots (-1: key 0)
  __shared__ int32_t ncomp, zmin, zcnt, zgroup;
  const int tid = threadIdx.x;
  for (int t = tid; t < kHashSlots; t += kSmallThreads) {
    hk[t] = 0ull;
    hmin[t] = 0x7FFFFFFF;
    hcnt[t] = 0;
  }
  if (tid == 0) {
    ncomp = 0;
    zmin = 0x7FFFFFFF;
    zcnt = 0;
  }
  __syncthreads();
  int myslot[kHashPer];
#pragma unroll
  for (int e = 0; e < kHashPer; ++e) {
    const int p = tid + e * kSmallThreads;
    myslot[e] = -1;
    if (p < R) {
      const unsigned long long m = map_key(keys[p]);
      if (m == 0ull) {
        atomicMin(&zmin, p);
        atomicAdd(&zcnt, 1);
      } else {
        uint32_t sl = (uint32_t)((m * 0x9E3779B97F4A7C15ull) >> 52) & (kHashSlots - 1);
        for (;;) {   // at most R probes: fewer keys than slots
          const unsigned long long prev = atomicCAS(&hk[sl], 0ull, m);
          if (prev == 0ull || prev == m) break;
          sl = (sl + 1) & (kHashSlots - 1);
        }
        atomicMin(&hmin[sl], p);
        atomicAdd(&hcnt[sl], 1);
        myslot[e] = (int)sl;
      }
    }
  }
  __syncthreads();
  // distinct keys in slot order
  for (int t = tid; t < kHashSlots; t += kSmallThreads) {
    if (hk[t] != 0ull) {
      const int u = atomicAdd(&ncomp, 1);
      ck[u] = hk[t];
      cslot[u] = t;
    }
  }
  __syncthreads();
  if (tid == 0 && zcnt > 0) {
    ck[ncomp] = 0ull;
    cslot[ncomp] = -1;
    ++ncomp;
  }
  __syncthreads();
  const int n = ncomp;
  // group id = number of distinct keys below (keys are distinct); the list
  // is padded to a multiple of 8 with all-ones keys (never below a key) so
  // that eight independent reads are in flight at a time
  const int n8 = (n + 7) & ~7;
  for (int u = n + tid; u < n8; u += kSmallThreads) ck[u] = ~0ull;
  __syncthreads();
  for (int u = tid; u < n; u += kSmallThreads) {
    const unsigned long long m = ck[u];
    int r = 0;
    for (int j = 0; j < n8; j += 8) {
      unsigned long long b[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) b[t] = ck[j + t];
#pragma unroll
      for (int t = 0; t < 8; ++t) r += b[t] < m ? 1 : 0;
    }
    const int sl = cslot[u];
    uk[r] = unmap_key(m);
    if (sl >= 0) {
      fi[r] = hmin[sl];
      if (cnt) cnt[r] = hcnt[sl];
      hmin[sl] = r;   // (this thread is the only one that reads the slot here)
    } else {
      fi[r] = zmin;
      if (cnt) cnt[r] = zcnt;
      zgroup = r;
    }
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < kHashPer; ++e) {
    const int p = tid + e * kSmallThreads;
    if (p < R) inv[p] = myslot[e] >= 0 ? hmin[myslot[e]] : zgroup;
  }
  if (tid == 0) *nu_out = (int64_t)n;
}

// ---------------------------------------------------------------- radix path

struct RadixWs {
  uint64_t *keyA, *keyB;
  int32_t *idxA, *idxB;
  uint64_t *pmin, *pmax;   // per-block min/max of mapped keys
  uint64_t *range;         // [0] = global min, [1] = radix pass count,
                           // [2] = key values of the dense path (0: radix)
  uint32_t *hist;          // kBins x nb, digit-major
  uint32_t *bheads;        // heads per block
  int32_t *start;          // group start positions
};

__global__ __launch_bounds__(kRadixThreads) void radix_prep_kernel(
    const int64_t *__restrict__ keys, int R, RadixWs ws) {
  __shared__ uint64_t smin[kRadixThreads / 64], smax[kRadixThreads / 64];
  const int b = blockIdx.x, tid = threadIdx.x;
  uint64_t mn = ~0ull, mx = 0ull;
  for (int e = 0; e < kRadixItems; ++e) {
    int p = b * kTile + e * kRadixThreads + tid;
    if (p < R) {
      uint64_t k = map_key(keys[p]);
      ws.keyA[p] = k;
      ws.idxA[p] = p;
      mn = k < mn ? k : mn;
      mx = k > mx ? k : mx;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t a = __shfl_xor(mn, o, 64), c = __shfl_xor(mx, o, 64);
    mn = a < mn ? a : mn;
    mx = c > mx ? c : mx;
  }
  if ((tid & 63) == 0) {
    smin[tid >> 6] = mn;
    smax[tid >> 6] = mx;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kRadixThreads / 64; ++w) {
      mn = smin[w] < mn ? smin[w] : mn;
      mx = smax[w] > mx ? smax[w] : mx;
    }
    ws.pmin[b] = mn;
    ws.pmax[b] = mx;
  }
}

__global__ __launch_bounds__(1024) void radix_range_kernel(int R, int nb, RadixWs ws) {
  __shared__ uint64_t smin[16], smax[16];
  const int tid = threadIdx.x;
  uint64_t mn = ~0ull, mx = 0ull;
  for (int i = tid; i < nb; i += 1024) {
    mn = ws.pmin[i] < mn ? ws.pmin[i] : mn;
    mx = ws.pmax[i] > mx ? ws.pmax[i] : mx;
  }
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t a = __shfl_xor(mn, o, 64), c = __shfl_xor(mx, o, 64);
    mn = a < mn ? a : mn;
    mx = c > mx ? c : mx;
  }
  if ((tid & 63) == 0) {
    smin[tid >> 6] = mn;
    smax[tid >> 6] = mx;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < 16; ++w) {
      mn = smin[w] < mn ? smin[w] : mn;
      mx = smax[w] > mx ? smax[w] : mx;
    }
    uint64_t span = mx - mn;
    int bits = span ? 64 - __clzll((long long)span) : 0;
    // dense path when the keys take at most R values
    const bool dense = span < (uint64_t)R;
    ws.range[0] = mn;
    ws.range[1] = dense ? 0ull : (uint64_t)((bits + kRadixBits - 1) / kRadixBits);
    ws.range[2] = dense ? span + 1 : 0ull;
  }
}

__device__ __forceinline__ uint32_t digit_of(uint64_t k, uint64_t mn, int pass) {
  return (uint32_t)(((k - mn) >> (pass * kRadixBits)) & (kBins - 1));
}

__global__ __launch_bounds__(kRadixThreads) void radix_hist_kernel(int R, int nb, int pass,
                                                                   RadixWs ws) {
  __shared__ uint32_t h[kBins];
  const uint64_t npass = ws.range[1];
  if ((uint64_t)pass >= npass) return;
  const uint64_t mn = ws.range[0];
  const uint64_t *src = (pass & 1) ? ws.keyB : ws.keyA;
  const int b = blockIdx.x, tid = threadIdx.x;
  h[tid] = 0;
  __syncthreads();
  for (int e = 0; e < kRadixItems; ++e) {
    int p = b * kTile + e * kRadixThreads + tid;
    if (p < R) atomicAdd(&h[digit_of(src[p], mn, pass)], 1u);
  }
  __syncthreads();
  ws.hist[tid * nb + b] = h[tid];
}

__global__ __launch_bounds__(kRadixThreads) void radix_scatter_kernel(int R, int nb, int pass,
                                                                      RadixWs ws) {
  __shared__ uint32_t goff[kBins];
  __shared__ uint32_t running[kBins];
  __shared__ uint32_t wcount[kRadixThreads / 64][kBins];
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  const uint64_t npass = ws.range[1];
  if ((uint64_t)pass >= npass) return;
  const uint64_t mn = ws.range[0];
  const uint64_t *ksrc = (pass & 1) ? ws.keyB : ws.keyA;
  uint64_t *kdst = (pass & 1) ? ws.keyA : ws.keyB;
  const int32_t *isrc = (pass & 1) ? ws.idxB : ws.idxA;
  int32_t *idst = (pass & 1) ? ws.idxA : ws.idxB;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

  // global base of each digit for this block: all smaller digits everywhere,
  // plus this digit in earlier blocks
  uint32_t tot = 0, prior = 0;
  for (int bb = 0; bb < nb; ++bb) {
    uint32_t c = ws.hist[tid * nb + bb];
    tot += c;
    if (bb < b) prior += c;
  }
  uint32_t total;
  uint32_t incl = block_inclusive_scan<kRadixThreads>(tot, wsum, total);
  goff[tid] = incl - tot + prior;
  running[tid] = 0;
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int e = 0; e < kRadixItems; ++e) {
    for (int i = tid; i < (kRadixThreads / 64) * kBins; i += kRadixThreads)
      (&wcount[0][0])[i] = 0;
    __syncthreads();
    int p = b * kTile + e * kRadixThreads + tid;
    bool valid = p < R;
    uint64_t key = valid ? ksrc[p] : 0ull;
    int32_t idx = valid ? isrc[p] : 0;
    uint32_t d = valid ? digit_of(key, mn, pass) : 0u;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < kRadixBits; ++bit) {
      bool s = (d >> bit) & 1u;
      uint64_t bal = __ballot(s);
      peers &= s ? bal : ~bal;
    }
    uint32_t rank = (uint32_t)__popcll(peers & lt);
    if (valid && rank == 0) wcount[w][d] = (uint32_t)__popcll(peers);
    __syncthreads();
    if (valid) {
      uint32_t pos = goff[d] + running[d] + rank;
      for (int ww = 0; ww < w; ++ww) pos += wcount[ww][d];
      if (pos < (uint32_t)R) {  // always true for a consistent histogram
        kdst[pos] = key;
        idst[pos] = idx;
      }
    }
    __syncthreads();
    uint32_t add = 0;
    for (int ww = 0; ww < kRadixThreads / 64; ++ww) add += wcount[ww][tid];
    running[tid] += add;
    __syncthreads();
  }
}

__device__ __forceinline__ const uint64_t *sorted_keys(const RadixWs &ws) {
  return (ws.range[1] & 1) ? ws.keyB : ws.keyA;
}
__device__ __forceinline__ const int32_t *sorted_idx(const RadixWs &ws) {
  return (ws.range[1] & 1) ? ws.idxB : ws.idxA;
}

__global__ __launch_bounds__(kRadixThreads) void radix_heads_kernel(int R, RadixWs ws) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  if (ws.range[2]) return;   // dense path
  const uint64_t *k = sorted_keys(ws);
  const int b = blockIdx.x, tid = threadIdx.x;
  uint32_t h = 0;
  for (int e = 0; e < kRadixItems; ++e) {
    int p = b * kTile + e * kRadixThreads + tid;
    if (p < R) h += (p == 0 || k[p] != k[p - 1]) ? 1u : 0u;
  }
  uint32_t total;
  block_inclusive_scan<kRadixThreads>(h, wsum, total);
  if (tid == 0) ws.bheads[b] = total;
}

__global__ __launch_bounds__(kRadixThreads) void radix_compact_kernel(
    int R, RadixWs ws, int64_t *__restrict__ uk, int32_t *__restrict__ fi,
    int32_t *__restrict__ inv, int64_t *__restrict__ nu_out) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  if (ws.range[2]) return;   // dense path
  const uint64_t *k = sorted_keys(ws);
  const int32_t *ix = sorted_idx(ws);
  const int b = blockIdx.x, tid = threadIdx.x;
  uint32_t before = 0;
  for (int bb = tid; bb < b; bb += kRadixThreads) before += ws.bheads[bb];
  uint32_t g0;  // heads in all earlier blocks
  block_inclusive_scan<kRadixThreads>(before, wsum, g0);
  // thread t owns positions [base + t*I, base + t*I + I) so that the scan
  // order is the sorted order
  const int base = b * kTile + tid * kRadixItems;
  uint32_t h = 0;
  for (int e = 0; e < kRadixItems; ++e) {
    int p = base + e;
    if (p < R) h += (p == 0 || k[p] != k[p - 1]) ? 1u : 0u;
  }
  uint32_t total;
  uint32_t incl = block_inclusive_scan<kRadixThreads>(h, wsum, total);
  uint32_t g = g0 + incl - h;
  for (int e = 0; e < kRadixItems; ++e) {
    int p = base + e;
    if (p >= R) break;
    uint64_t kk = k[p];
    const int32_t src = ix[p];
    if (p == 0 || kk != k[p - 1]) {
      if (g < (uint32_t)R) {
        uk[g] = unmap_key(kk);
        fi[g] = src;
        ws.start[g] = p;
      }
      ++g;
    }
    if ((uint32_t)src < (uint32_t)R) inv[src] = (int32_t)(g - 1);
    if (p == R - 1) {
      *nu_out = (int64_t)g;
      if (g <= (uint32_t)R) ws.start[g] = R;
    }
  }
}

__global__ __launch_bounds__(256) void radix_counts_kernel(int R, RadixWs ws,
                                                           const int64_t *__restrict__ nu,
                                                           int32_t *__restrict__ cnt) {
  if (ws.range[2]) return;   // dense path
  int g = blockIdx.x * 256 + threadIdx.x;
  if (g < R && (int64_t)g < *nu) cnt[g] = ws.start[g + 1] - ws.start[g];
}

// ---------------------------------------------------------------- dense path
//
// When the R mapped keys take at most R values (max - min < R: e.g. chunk
// row ids), the groups are found by direct addressing over [min, max]
// instead of sorting: per key value v, the first request (atomic min) and the
// group size (atomic add); a scan over the values numbers the present ones
// in ascending key order; each request then reads its group.  Same canonical
// outputs as the sort.  Value arrays reuse the sort's second buffers:
// first/count in keyB (2 x int32 per value), group ids in idxB; the scan's
// block sums use the histogram buffer.

constexpr int kDenseBlk = 1024;                  // values per scan block
constexpr int kAggRound = 1024, kAggSlots = 2048;

__device__ __forceinline__ int32_t *dense_first(const RadixWs &ws) { return (int32_t *)ws.keyB; }
__device__ __forceinline__ int32_t *dense_count(const RadixWs &ws, uint64_t nv) {
  return (int32_t *)ws.keyB + nv;
}

__global__ void dense_clear_kernel(RadixWs ws) {
  const uint64_t nv = ws.range[2];
  if (!nv) return;
  int32_t *first = dense_first(ws), *count = dense_count(ws, nv);
  for (uint64_t v = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; v < nv;
       v += (uint64_t)gridDim.x * blockDim.x) {
    first[v] = 0x7fffffff;
    count[v] = 0;
  }
}

// Rounds of kAggRound consecutive requests are first combined per key value
// in an LDS table (a hot key appears many times per round), then each table
// entry goes to the value arrays with one atomic min and one atomic add.
__global__ __launch_bounds__(256) void dense_mark_kernel(int R, RadixWs ws) {
  __shared__ int32_t tkey[kAggSlots];
  __shared__ int32_t tfirst[kAggSlots];
  __shared__ int32_t tcount[kAggSlots];
  const uint64_t nv = ws.range[2];
  if (!nv) return;
  const uint64_t mn = ws.range[0];
  int32_t *first = dense_first(ws), *count = dense_count(ws, nv);
  const int tid = threadIdx.x;
  for (int64_t r0 = (int64_t)blockIdx.x * kAggRound; r0 < R;
       r0 += (int64_t)gridDim.x * kAggRound) {
    for (int j = tid; j < kAggSlots; j += 256) {
      tkey[j] = -1;
      tfirst[j] = 0x7fffffff;
      tcount[j] = 0;
    }
    __syncthreads();
    for (int j = tid; j < kAggRound; j += 256) {
      const int64_t p = r0 + j;
      if (p >= R) break;
      const int32_t v = (int32_t)(ws.keyA[p] - mn);   // < nv <= R
      uint32_t h = ((uint32_t)v * 2654435761u) & (kAggSlots - 1);
      for (;;) {   // at most kAggRound keys in kAggSlots slots: a slot is found
        const int32_t prev = atomicCAS(&tkey[h], -1, v);
        if (prev == -1 || prev == v) break;
        h = (h + 1) & (kAggSlots - 1);
      }
      atomicMin(&tfirst[h], (int32_t)p);
      atomicAdd(&tcount[h], 1);
    }
    __syncthreads();
    for (int j = tid; j < kAggSlots; j += 256) {
      const int32_t v = tkey[j];
      if (v >= 0) {
        atomicMin(&first[v], tfirst[j]);
        atomicAdd(&count[v], tcount[j]);
      }
    }
    __syncthreads();
  }
}

// Present values per scan block.
__global__ __launch_bounds__(kDenseBlk) void dense_blocksum_kernel(RadixWs ws) {
  __shared__ uint32_t wsum[kDenseBlk / 64 + 1];
  const uint64_t nv = ws.range[2];
  if (!nv || (uint64_t)blockIdx.x * kDenseBlk >= nv) return;
  const int32_t *count = dense_count(ws, nv);
  const uint64_t v = (uint64_t)blockIdx.x * kDenseBlk + threadIdx.x;
  const uint32_t pr = v < nv && count[v] > 0 ? 1u : 0u;
  uint32_t total;
  block_inclusive_scan<kDenseBlk>(pr, wsum, total);
  if (threadIdx.x == 0) ws.hist[blockIdx.x] = total;
}

// Group numbers of the present values (ascending), and the per-group outputs.
__global__ __launch_bounds__(kDenseBlk) void dense_groups_kernel(
    RadixWs ws, int64_t *__restrict__ uk, int32_t *__restrict__ fi, int32_t *__restrict__ cnt,
    int64_t *__restrict__ nu_out) {
  __shared__ uint32_t wsum[kDenseBlk / 64 + 1];
  const uint64_t nv = ws.range[2];
  if (!nv || (uint64_t)blockIdx.x * kDenseBlk >= nv) return;
  const uint64_t mn = ws.range[0];
  const int32_t *first = dense_first(ws), *count = dense_count(ws, nv);
  int32_t *gid = ws.idxB;
  const int b = blockIdx.x, tid = threadIdx.x;
  uint32_t before = 0;   // present values in all earlier blocks
  for (int bb = tid; bb < b; bb += kDenseBlk) before += ws.hist[bb];
  uint32_t g0;
  block_inclusive_scan<kDenseBlk>(before, wsum, g0);
  const uint64_t v = (uint64_t)b * kDenseBlk + tid;
  const uint32_t pr = v < nv && count[v] > 0 ? 1u : 0u;
  uint32_t total;
  const uint32_t incl = block_inclusive_scan<kDenseBlk>(pr, wsum, total);
  if (pr) {
    const uint32_t g = g0 + incl - 1u;
    uk[g] = unmap_key(mn + v);
    fi[g] = first[v];
    if (cnt) cnt[g] = count[v];
    gid[v] = (int32_t)g;
  }
  if ((uint64_t)(b + 1) * kDenseBlk >= nv && tid == 0) *nu_out = (int64_t)(g0 + total);
}

__global__ void dense_inverse_kernel(int R, RadixWs ws, int32_t *__restrict__ inv) {
  const uint64_t nv = ws.range[2];
  if (!nv) return;
  const uint64_t mn = ws.range[0];
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < R;
       p += (int64_t)gridDim.x * blockDim.x)
    inv[p] = ws.idxB[ws.keyA[p] - mn];
}

// ---------------------------------------------------------------- host side

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

size_t dedup_workspace_bytes(int64_t R) {
  if (R <= kSmallMax) return 0;
  size_t nb = (size_t)((R + kTile - 1) / kTile);
  size_t s = 0;
  s += 2 * align_up(sizeof(uint64_t) * R);
  s += 2 * align_up(sizeof(int32_t) * R);
  s += 2 * align_up(sizeof(uint64_t) * nb);
  s += align_up(sizeof(uint64_t) * 4);
  s += align_up(sizeof(uint32_t) * kBins * nb);
  s += align_up(sizeof(uint32_t) * nb);
  s += align_up(sizeof(int32_t) * (R + 1));
  return s;
}

hipError_t launch_dedup(const int64_t *keys, int64_t R, int64_t *uk, int32_t *fi, int32_t *cnt,
                        int32_t *inv, int64_t *nu, void *ws, hipStream_t st) {
  if (R <= kHashMax) {
    hipLaunchKernelGGL(dedup_hash_kernel, dim3(1), dim3(kSmallThreads), 0, st, keys, (int)R, uk,
                       fi, cnt, inv, nu);
    return hipGetLastError();
  }
  if (R <= kSmallMax) {
    int P = 1;
    while (P < R) P <<= 1;
    if (P < 2) P = 2;
    hipLaunchKernelGGL(dedup_small_kernel, dim3(1), dim3(kSmallThreads), 0, st, keys, (int)R,
                       P, uk, fi, cnt, inv, nu);
    return hipGetLastError();
  }
  const int nb = (int)((R + kTile - 1) / kTile);
  char *p = (char *)ws;
  RadixWs w;
  w.keyA = (uint64_t *)p; p += align_up(sizeof(uint64_t) * R);
  w.keyB = (uint64_t *)p; p += align_up(sizeof(uint64_t) * R);
  w.idxA = (int32_t *)p; p += align_up(sizeof(int32_t) * R);
  w.idxB = (int32_t *)p; p += align_up(sizeof(int32_t) * R);
  w.pmin = (uint64_t *)p; p += align_up(sizeof(uint64_t) * nb);
  w.pmax = (uint64_t *)p; p += align_up(sizeof(uint64_t) * nb);
  w.range = (uint64_t *)p; p += align_up(sizeof(uint64_t) * 4);
  w.hist = (uint32_t *)p; p += align_up(sizeof(uint32_t) * kBins * nb);
  w.bheads = (uint32_t *)p; p += align_up(sizeof(uint32_t) * nb);
  w.start = (int32_t *)p;
  hipLaunchKernelGGL(radix_prep_kernel, dim3(nb), dim3(kRadixThreads), 0, st, keys, (int)R, w);
  hipLaunchKernelGGL(radix_range_kernel, dim3(1), dim3(1024), 0, st, (int)R, nb, w);
  // dense path (each kernel returns at once when the keys need the sort)
  {
    const unsigned vb = (unsigned)((R + kDenseBlk - 1) / kDenseBlk);   // nv <= R
    hipLaunchKernelGGL(dense_clear_kernel, dim3(vb), dim3(kDenseBlk), 0, st, w);
    hipLaunchKernelGGL(dense_mark_kernel, dim3((unsigned)((R + kAggRound - 1) / kAggRound)),
                       dim3(256), 0, st, (int)R, w);
    hipLaunchKernelGGL(dense_blocksum_kernel, dim3(vb), dim3(kDenseBlk), 0, st, w);
    hipLaunchKernelGGL(dense_groups_kernel, dim3(vb), dim3(kDenseBlk), 0, st, w, uk, fi, cnt, nu);
    hipLaunchKernelGGL(dense_inverse_kernel, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, st,
                       (int)R, w, inv);
  }
  for (int pass = 0; pass < 64 / kRadixBits; ++pass) {
    hipLaunchKernelGGL(radix_hist_kernel, dim3(nb), dim3(kRadixThreads), 0, st, (int)R, nb,
                       pass, w);
    hipLaunchKernelGGL(radix_scatter_kernel, dim3(nb), dim3(kRadixThreads), 0, st, (int)R, nb,
                       pass, w);
  }
  hipLaunchKernelGGL(radix_heads_kernel, dim3(nb), dim3(kRadixThreads), 0, st, (int)R, w);
  hipLaunchKernelGGL(radix_compact_kernel, dim3(nb), dim3(kRadixThreads), 0, st, (int)R, w, uk,
                     fi, inv, nu);
  if (cnt) {
    hipLaunchKernelGGL(radix_counts_kernel, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, st,
                       (int)R, w, (const int64_t *)nu, cnt);
  }
  return hipGetLastError();
}

}  // namespace hs
