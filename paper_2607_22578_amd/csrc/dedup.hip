// Step 1: signature matching -- group R request keys.
//
// HeraSys Sec. 3.3 (I): a node whose signature matches a node already in the
// window is fused into it; Eq. (3) aggregates over the merged set M(v*).  The
// paper detects matches with a hash map (Appendix B.3, Phase 1).  On the GPU
// every path below gives the same canonical outputs (those of a stable sort
// of (key, request) pairs): distinct keys ascending, the survivor of a group
// is its earliest request, counts[g] = |M(v*)|, inverse[i] = group.
//
// Three paths:
//   R <= kHashMax  : one workgroup groups the keys in an LDS hash table
//                    (first request by atomic min, group size by atomic add),
//                    orders the distinct keys by counting, for each, the
//                    distinct keys below it, and maps every request to its
//                    group through the table;
//   R <= kSmallMax : one workgroup sorts (key, idx) in LDS with a bitonic
//                    network and compacts in the same launch;
//   larger R       : the key range is found on the device; keys that take at
//                    most R values are grouped by direct addressing over the
//                    range, others by an LSD radix sort (8-bit digits over
//                    key - min, so only the bits that vary are sorted; stable
//                    local ranking with wavefront ballots, then head flags, a
//                    compaction and group sizes) in one persistent launch.
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

// ---------------------------------------------------------------- larger R
//
// Five launches whatever the keys:
//   prep    : mapped keys and request numbers, per-workgroup key min/max, and
//             the scratch the later launches need at its neutral value;
//   mark    : every workgroup reduces the min/max itself and picks the path;
//             dense path (the keys take at most R values, max - min < R):
//             first request and group size per key value;
//   groups  : dense path: the present values numbered in ascending order by
//             a single-pass scan (each value block looks back at the running
//             totals of the blocks before it), with the per-group outputs;
//   inverse : dense path: request -> group;
//   radix   : sort path (returns at once on the dense path): one persistent
//             launch of at most kRadixGridMax workgroups, all resident, that
//             runs every LSD pass (8-bit digits of key - min, one pass per
//             8 bits of max - min), then head flags, compaction and group
//             sizes, with grid barriers between the phases.
// The three dense launches return at once on the sort path.

constexpr int kPrepMax = 1024;        // prep workgroups (min/max partials)
constexpr int kRadixGridMax = 256;    // workgroups of the persistent sort
constexpr int kBarGroups = 16;        // arrival counters of the grid barrier
constexpr int kCtlStride = 32;        // 32-bit words between counters (128 B)
// control words: [0] value-block ticket of the groups launch; barrier
// arrival counter j at (1 + j) * kCtlStride; the barrier's release counter at
// (1 + kBarGroups) * kCtlStride
constexpr int kCtlWords = (2 + kBarGroups) * kCtlStride;

struct RadixWs {
  uint64_t *keyA, *keyB;
  int32_t *idxA, *idxB;
  uint64_t *pmin, *pmax;   // per-prep-workgroup min/max of mapped keys
  uint64_t *range;         // [0] = global min, [1] = radix pass count,
                           // [2] = key values of the dense path (0: radix)
  uint32_t *hist;          // kBins x nb, digit-major (scanned in place)
  uint32_t *dtot;          // kBins digit totals of a pass
  uint32_t *bheads;        // heads per tile (scanned in place)
  int32_t *start;          // group start positions
  uint64_t *flags;         // dense value blocks: running-total words
  uint32_t *ctl;           // kCtlWords control words
};

// ------------------------------------------------ grid-wide helpers

// Barrier over the G workgroups of a launch that are all resident at once
// (G at most what the device holds of them).  `k`
// counts the barriers this workgroup has passed (the counters only grow
// within a launch; prep zeroes them).  Arrivals are spread over kBarGroups
// counters so that no single address takes all G of them; the last arrival
// of each group bumps the release counter that everyone waits on.
__device__ __forceinline__ void grid_barrier(uint32_t *ctl, int G, uint32_t &k) {
  ++k;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    const int ng = G < kBarGroups ? G : kBarGroups;
    const int j = (int)blockIdx.x % ng;
    const uint32_t gsize = (uint32_t)(G / ng + (j < G % ng ? 1 : 0));
    uint32_t *sub = ctl + (1 + j) * kCtlStride;
    uint32_t *rel = ctl + (1 + kBarGroups) * kCtlStride;
    const uint32_t old =
        __hip_atomic_fetch_add(sub, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == k * gsize)
      __hip_atomic_fetch_add(rel, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    while (__hip_atomic_load(rel, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < k * (uint32_t)ng)
      __builtin_amdgcn_s_sleep(1);
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Exclusive prefix sum of a[0, n) in place by one workgroup; returns the
// total.
__device__ uint32_t block_scan_inplace(uint32_t *a, int64_t n) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  constexpr int P = 4;
  uint32_t carry = 0;
  for (int64_t c0 = 0; c0 < n; c0 += kRadixThreads * P) {
    const int64_t i0 = c0 + (int64_t)threadIdx.x * P;
    uint32_t v[P], sum = 0;
#pragma unroll
    for (int e = 0; e < P; ++e) {
      v[e] = i0 + e < n ? a[i0 + e] : 0u;
      sum += v[e];
    }
    uint32_t total;
    uint32_t run = carry + block_inclusive_scan<kRadixThreads>(sum, wsum, total) - sum;
#pragma unroll
    for (int e = 0; e < P; ++e)
      if (i0 + e < n) {
        a[i0 + e] = run;
        run += v[e];
      }
    carry += total;
  }
  return carry;
}

// ------------------------------------------------ prep and path choice

// Workgroup b of P: chunks of kPrepChunk requests b, b + P, ... -> mapped
// keys (keyA), request numbers (idxA) and the min/max over them; the dense
// tables for up to R values, the value-block words and the control words to
// their neutral values.
constexpr int kPrepChunk = 4 * kRadixThreads;
__global__ __launch_bounds__(kRadixThreads) void dedup_prep_kernel(
    const int64_t *__restrict__ keys, int R, RadixWs ws) {
  __shared__ uint64_t smin[kRadixThreads / 64], smax[kRadixThreads / 64];
  const int tid = threadIdx.x, P = gridDim.x;
  uint64_t mn = ~0ull, mx = 0ull;
  for (int64_t c = blockIdx.x; c * kPrepChunk < R; c += P) {
#pragma unroll
    for (int e = 0; e < kPrepChunk / kRadixThreads; ++e) {
      const int64_t p = c * kPrepChunk + e * kRadixThreads + tid;
      if (p < R) {
        const uint64_t k = map_key(keys[p]);
        ws.keyA[p] = k;
        ws.idxA[p] = (int32_t)p;
        mn = k < mn ? k : mn;
        mx = k > mx ? k : mx;
      }
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
    ws.pmin[blockIdx.x] = mn;
    ws.pmax[blockIdx.x] = mx;
  }
  // dense tables (first request, group size) over [0, R) >= [0, nv)
  int32_t *first = (int32_t *)ws.keyB, *count = (int32_t *)ws.keyB + R;
  const int64_t gt = (int64_t)blockIdx.x * kRadixThreads + tid;
  const int64_t gs = (int64_t)P * kRadixThreads;
  for (int64_t v = gt; v < R; v += gs) {
    first[v] = 0x7fffffff;
    count[v] = 0;
  }
  const int64_t nvb = ((int64_t)R + 1023) / 1024;
  for (int64_t i = gt; i < nvb; i += gs) ws.flags[i] = 0ull;
  if (blockIdx.x == 0)
    for (int i = tid; i < kCtlWords; i += kRadixThreads) ws.ctl[i] = 0u;
}

struct Range {
  uint64_t mn;
  uint64_t npass;   // radix passes (0 on the dense path)
  uint64_t nv;      // key values of the dense path (0: radix path)
};

// Global min/max over the P prep partials and the path: dense when the keys
// take at most R values (max - min < R), else radix with one pass per 8 bits
// of max - min.  Computed by every workgroup that calls it.
__device__ Range range_of(int R, int P, const RadixWs &ws) {
  __shared__ uint64_t smin[kRadixThreads / 64], smax[kRadixThreads / 64];
  __shared__ Range res;
  const int tid = threadIdx.x;
  uint64_t mn = ~0ull, mx = 0ull;
  for (int i = tid; i < P; i += kRadixThreads) {
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
    for (int w = 1; w < kRadixThreads / 64; ++w) {
      mn = smin[w] < mn ? smin[w] : mn;
      mx = smax[w] > mx ? smax[w] : mx;
    }
    const uint64_t span = mx - mn;
    const int bits = span ? 64 - __clzll((long long)span) : 0;
    const bool dense = span < (uint64_t)R;
    res.mn = mn;
    res.npass = dense ? 0ull : (uint64_t)((bits + kRadixBits - 1) / kRadixBits);
    res.nv = dense ? span + 1 : 0ull;
  }
  __syncthreads();
  return res;
}

// ---------------------------------------------------------------- dense path
//
// When the R mapped keys take at most R values (e.g. chunk row ids), the
// groups are found by direct addressing over [min, max] instead of sorting:
// per key value v, the first request (atomic min) and the group size (atomic
// add); a scan over the values numbers the present ones in ascending key
// order; each request then reads its group.  Same canonical outputs as the
// sort.  Value arrays reuse the sort's second buffers: first/count in keyB
// (2 x int32 per value), group ids in idxB.

constexpr int kDenseBlk = 1024;                        // values per value block
constexpr int kDensePer = kDenseBlk / kRadixThreads;   // values per thread
constexpr int kAggRound = 1024, kAggSlots = 2048;

// Rounds of kAggRound consecutive requests are first combined per key value
// in an LDS table (a hot key appears many times per round), then each table
// entry goes to the value arrays with one atomic min and one atomic add.
// Workgroup 0 also stores the path for the later launches.
__global__ __launch_bounds__(kRadixThreads) void dense_mark_kernel(int R, int P, RadixWs ws) {
  __shared__ int32_t tkey[kAggSlots];
  __shared__ int32_t tfirst[kAggSlots];
  __shared__ int32_t tcount[kAggSlots];
  const Range rg = range_of(R, P, ws);
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid == 0) {
    ws.range[0] = rg.mn;
    ws.range[1] = rg.npass;
    ws.range[2] = rg.nv;
  }
  if (!rg.nv) return;
  int32_t *first = (int32_t *)ws.keyB, *count = (int32_t *)ws.keyB + R;
  for (int64_t round = blockIdx.x; round * kAggRound < R; round += gridDim.x) {
    const int64_t base = round * kAggRound;
    for (int j = tid; j < kAggSlots; j += kRadixThreads) {
      tkey[j] = -1;
      tfirst[j] = 0x7fffffff;
      tcount[j] = 0;
    }
    __syncthreads();
    for (int j = tid; j < kAggRound; j += kRadixThreads) {
      const int64_t p = base + j;
      if (p >= R) break;
      const int32_t v = (int32_t)(ws.keyA[p] - rg.mn);   // < nv <= R
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
    for (int j = tid; j < kAggSlots; j += kRadixThreads) {
      const int32_t v = tkey[j];
      if (v >= 0) {
        atomicMin(&first[v], tfirst[j]);
        atomicAdd(&count[v], tcount[j]);
      }
    }
    __syncthreads();
  }
}

// Value-block words: state in the high half (1: the block's own count, 2:
// the running total through the block), the number in the low half.
constexpr uint64_t kFlagAgg = 1ull << 32, kFlagPrefix = 2ull << 32;

// One value block per workgroup, in the order the workgroups start (a ticket,
// so every block it waits on has started): count the present values, publish
// the count, add up the counts or running totals of the blocks before it,
// publish the running total, then number its present values and write the
// per-group outputs.  The last block writes n_u.
__global__ __launch_bounds__(kRadixThreads) void dense_groups_kernel(
    int R, RadixWs ws, int64_t *__restrict__ uk, int32_t *__restrict__ fi,
    int32_t *__restrict__ cnt, int64_t *__restrict__ nu_out) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  __shared__ uint32_t s_vb, s_before;
  const uint64_t nv = ws.range[2];
  const uint64_t nvb = (nv + kDenseBlk - 1) / kDenseBlk;
  if (!nv || blockIdx.x >= nvb) return;
  const int tid = threadIdx.x;
  if (tid == 0)
    s_vb = __hip_atomic_fetch_add(ws.ctl, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  const uint64_t vb = s_vb;
  const uint64_t mn = ws.range[0];
  const int32_t *first = (const int32_t *)ws.keyB, *count = (const int32_t *)ws.keyB + R;
  int32_t *gid = ws.idxB;
  const uint64_t v0 = vb * kDenseBlk + (uint64_t)tid * kDensePer;
  int32_t c[kDensePer];
  uint32_t pr = 0;
#pragma unroll
  for (int e = 0; e < kDensePer; ++e) {
    c[e] = v0 + e < nv ? count[v0 + e] : 0;
    pr += c[e] > 0 ? 1u : 0u;
  }
  uint32_t total;
  const uint32_t incl = block_inclusive_scan<kRadixThreads>(pr, wsum, total);
  if (tid < 64) {
    // wave 0: publish this block's count, then add up the words of the
    // blocks before it, 64 at a time, back to the nearest running total
    // (blocks before the first count as a running total of 0)
    uint64_t *fl = ws.flags;
    const int lane = tid;
    uint32_t before = 0;
    if (vb == 0) {
      if (lane == 0)
        __hip_atomic_store(&fl[0], kFlagPrefix | total, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    } else {
      if (lane == 0)
        __hip_atomic_store(&fl[vb], kFlagAgg | total, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      for (int64_t j0 = (int64_t)vb - 1;; j0 -= 64) {
        const int64_t j = j0 - lane;
        uint64_t f = j >= 0 ? __hip_atomic_load(&fl[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                            : kFlagPrefix;
        while (__any(f == 0ull)) {
          __builtin_amdgcn_s_sleep(1);
          if (f == 0ull) f = __hip_atomic_load(&fl[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        const uint64_t pm = __ballot(f >= kFlagPrefix);
        const int stop = pm ? __ffsll((long long)pm) - 1 : 64;
        uint32_t v = lane <= stop ? (uint32_t)f : 0u;
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        before += v;
        if (pm) break;
      }
      if (lane == 0)
        __hip_atomic_store(&fl[vb], kFlagPrefix | (before + total), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    if (lane == 0) s_before = before;
  }
  __syncthreads();
  uint32_t g = s_before + incl - pr;
#pragma unroll
  for (int e = 0; e < kDensePer; ++e) {
    const uint64_t v = v0 + e;
    if (c[e] > 0) {
      uk[g] = unmap_key(mn + v);
      fi[g] = first[v];
      if (cnt) cnt[g] = c[e];
      gid[v] = (int32_t)g;
      ++g;
    }
  }
  if (vb + 1 == nvb && tid == 0) *nu_out = (int64_t)(s_before + total);
}

// Request -> group.
__global__ __launch_bounds__(256) void dense_inverse_kernel(int R, RadixWs ws,
                                                            int32_t *__restrict__ inv) {
  const uint64_t nv = ws.range[2];
  if (!nv) return;
  const uint64_t mn = ws.range[0];
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < R; p += (int64_t)gridDim.x * 256)
    inv[p] = ws.idxB[ws.keyA[p] - mn];
}

// ---------------------------------------------------------------- sort path

__device__ __forceinline__ uint32_t digit_of(uint64_t k, uint64_t mn, int pass) {
  return (uint32_t)(((k - mn) >> (pass * kRadixBits)) & (kBins - 1));
}

// Digit histogram of tile b for one pass.
__device__ __forceinline__ void hist_phase(int R, int nb, int pass, uint64_t mn, int b,
                                           const RadixWs &ws) {
  __shared__ uint32_t h[kBins];
  const uint64_t *src = (pass & 1) ? ws.keyB : ws.keyA;
  const int tid = threadIdx.x;
  h[tid] = 0;
  __syncthreads();
  for (int e = 0; e < kRadixItems; ++e) {
    int p = b * kTile + e * kRadixThreads + tid;
    if (p < R) atomicAdd(&h[digit_of(src[p], mn, pass)], 1u);
  }
  __syncthreads();
  ws.hist[tid * nb + b] = h[tid];
  __syncthreads();
}

// Stable scatter of tile b by its digit for one pass.  With at most
// kDirectTiles tiles the digit offsets come straight from the histogram;
// otherwise its rows are already exclusive scans over the tiles and dtot
// holds the digit totals.
constexpr int kDirectTiles = 64;
__device__ __forceinline__ void scatter_phase(int R, int nb, int pass, uint64_t mn, int b,
                                              const RadixWs &ws) {
  __shared__ uint32_t goff[kBins];
  __shared__ uint32_t running[kBins];
  __shared__ uint32_t wcount[kRadixThreads / 64][kBins];
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  const uint64_t *ksrc = (pass & 1) ? ws.keyB : ws.keyA;
  uint64_t *kdst = (pass & 1) ? ws.keyA : ws.keyB;
  const int32_t *isrc = (pass & 1) ? ws.idxB : ws.idxA;
  int32_t *idst = (pass & 1) ? ws.idxA : ws.idxB;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

  // global base of each digit for this tile: all smaller digits everywhere,
  // plus this digit in earlier tiles
  uint32_t tot, prior;
  if (nb <= kDirectTiles) {
    tot = 0;
    prior = 0;
    for (int bb = 0; bb < nb; ++bb) {
      const uint32_t c = ws.hist[tid * nb + bb];
      tot += c;
      prior += bb < b ? c : 0u;
    }
  } else {
    tot = ws.dtot[tid];
    prior = ws.hist[tid * nb + b];
  }
  uint32_t total;
  const uint32_t incl = block_inclusive_scan<kRadixThreads>(tot, wsum, total);
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

__device__ __forceinline__ const uint64_t *sorted_keys(const RadixWs &ws, uint64_t npass) {
  return (npass & 1) ? ws.keyB : ws.keyA;
}
__device__ __forceinline__ const int32_t *sorted_idx(const RadixWs &ws, uint64_t npass) {
  return (npass & 1) ? ws.idxB : ws.idxA;
}

// Group heads (first of each run of equal keys) in tile b of the sorted keys.
__device__ __forceinline__ void heads_phase(int R, uint64_t npass, int b, const RadixWs &ws) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  const uint64_t *k = sorted_keys(ws, npass);
  const int tid = threadIdx.x;
  uint32_t h = 0;
  for (int e = 0; e < kRadixItems; ++e) {
    int p = b * kTile + e * kRadixThreads + tid;
    if (p < R) h += (p == 0 || k[p] != k[p - 1]) ? 1u : 0u;
  }
  uint32_t total;
  block_inclusive_scan<kRadixThreads>(h, wsum, total);
  if (tid == 0) ws.bheads[b] = total;
}

// Distinct keys, survivors and the request -> group map from tile b; bheads
// holds the heads before each tile.
__device__ __forceinline__ void compact_phase(int R, uint64_t npass, int b, const RadixWs &ws,
                                              int64_t *__restrict__ uk, int32_t *__restrict__ fi,
                                              int32_t *__restrict__ inv,
                                              int64_t *__restrict__ nu_out) {
  __shared__ uint32_t wsum[kRadixThreads / 64 + 1];
  const uint64_t *k = sorted_keys(ws, npass);
  const int32_t *ix = sorted_idx(ws, npass);
  const int tid = threadIdx.x;
  const uint32_t g0 = ws.bheads[b];
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

// The whole sort path in one persistent launch of G workgroups (all resident
// at once): per pass a
// digit histogram per tile, with more than kDirectTiles tiles an exclusive
// scan of each digit's row over the tiles (rows spread over the wavefronts),
// and the stable scatter; then
// head counts per tile, their scan (workgroup 0), the compaction and the
// group sizes.  Tiles are taken b, b + G, ...; the barrier count is the same
// for every workgroup.
__global__ __launch_bounds__(kRadixThreads) void radix_sort_kernel(
    int R, int nb, RadixWs ws, int64_t *__restrict__ uk, int32_t *__restrict__ fi,
    int32_t *__restrict__ cnt, int32_t *__restrict__ inv, int64_t *__restrict__ nu_out) {
  if (ws.range[2]) return;   // dense path
  const uint64_t mn = ws.range[0], npass = ws.range[1];
  const int G = gridDim.x, b = blockIdx.x;
  uint32_t k = 0;
  const int wid = b * (kRadixThreads / 64) + (threadIdx.x >> 6), nw = G * (kRadixThreads / 64);
  const int lane = threadIdx.x & 63;
  for (int pass = 0; pass < (int)npass; ++pass) {
    for (int t = b; t < nb; t += G) hist_phase(R, nb, pass, mn, t, ws);
    grid_barrier(ws.ctl, G, k);
    if (nb > kDirectTiles) {
      // each digit's row: exclusive scan over the tiles by one wavefront
      for (int d = wid; d < kBins; d += nw) {
        uint32_t *row = ws.hist + (int64_t)d * nb;
        uint32_t carry = 0;
        for (int c0 = 0; c0 < nb; c0 += 4 * 64) {
          const int i0 = c0 + lane * 4;
          uint32_t v[4], sum = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = i0 + e < nb ? row[i0 + e] : 0u;
            sum += v[e];
          }
          uint32_t x = sum;
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
          }
          uint32_t run = carry + x - sum;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (i0 + e < nb) {
              row[i0 + e] = run;
              run += v[e];
            }
          carry += __shfl(x, 63, 64);
        }
        if (lane == 0) ws.dtot[d] = carry;
      }
      grid_barrier(ws.ctl, G, k);
    }
    for (int t = b; t < nb; t += G) scatter_phase(R, nb, pass, mn, t, ws);
    grid_barrier(ws.ctl, G, k);
  }
  for (int t = b; t < nb; t += G) heads_phase(R, npass, t, ws);
  grid_barrier(ws.ctl, G, k);
  if (b == 0) block_scan_inplace(ws.bheads, nb);
  grid_barrier(ws.ctl, G, k);
  for (int t = b; t < nb; t += G) compact_phase(R, npass, t, ws, uk, fi, inv, nu_out);
  if (cnt) {
    grid_barrier(ws.ctl, G, k);
    const int64_t n = *nu_out;
    for (int64_t g = (int64_t)b * kRadixThreads + threadIdx.x; g < R && g < n;
         g += (int64_t)G * kRadixThreads)
      cnt[g] = ws.start[g + 1] - ws.start[g];
  }
}

// ---------------------------------------------------------------- host side

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

size_t dedup_workspace_bytes(int64_t R) {
  if (R <= kSmallMax) return 0;
  size_t nb = (size_t)((R + kTile - 1) / kTile);
  size_t nvb = (size_t)((R + kDenseBlk - 1) / kDenseBlk);
  size_t s = 0;
  s += 2 * align_up(sizeof(uint64_t) * R);
  s += 2 * align_up(sizeof(int32_t) * R);
  s += 2 * align_up(sizeof(uint64_t) * kPrepMax);
  s += align_up(sizeof(uint64_t) * 4);
  s += align_up(sizeof(uint32_t) * kBins * nb);
  s += align_up(sizeof(uint32_t) * kBins);
  s += align_up(sizeof(uint32_t) * nb);
  s += align_up(sizeof(int32_t) * (R + 1));
  s += align_up(sizeof(uint64_t) * nvb);
  s += align_up(sizeof(uint32_t) * kCtlWords);
  return s;
}

// Workgroups of radix_sort_kernel that the current device holds at once (0:
// unknown).
static int radix_capacity() {
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev]) return cache[dev] > 0 ? cache[dev] : 0;
  int cus = 0, per = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, radix_sort_kernel, kRadixThreads, 0) !=
          hipSuccess ||
      cus <= 0 || per <= 0) {
    cache[dev] = -1;
    return 0;
  }
  cache[dev] = cus * per;
  return cache[dev];
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
  const int capacity = radix_capacity();
  if (capacity <= 0) return hipErrorNotSupported;
  const int nb = (int)((R + kTile - 1) / kTile);
  const int64_t nvb = (R + kDenseBlk - 1) / kDenseBlk;
  char *p = (char *)ws;
  RadixWs w;
  w.keyA = (uint64_t *)p; p += align_up(sizeof(uint64_t) * R);
  w.keyB = (uint64_t *)p; p += align_up(sizeof(uint64_t) * R);
  w.idxA = (int32_t *)p; p += align_up(sizeof(int32_t) * R);
  w.idxB = (int32_t *)p; p += align_up(sizeof(int32_t) * R);
  w.pmin = (uint64_t *)p; p += align_up(sizeof(uint64_t) * kPrepMax);
  w.pmax = (uint64_t *)p; p += align_up(sizeof(uint64_t) * kPrepMax);
  w.range = (uint64_t *)p; p += align_up(sizeof(uint64_t) * 4);
  w.hist = (uint32_t *)p; p += align_up(sizeof(uint32_t) * kBins * nb);
  w.dtot = (uint32_t *)p; p += align_up(sizeof(uint32_t) * kBins);
  w.bheads = (uint32_t *)p; p += align_up(sizeof(uint32_t) * nb);
  w.start = (int32_t *)p; p += align_up(sizeof(int32_t) * (R + 1));
  w.flags = (uint64_t *)p; p += align_up(sizeof(uint64_t) * nvb);
  w.ctl = (uint32_t *)p;
  int Ri = (int)R;
  const int64_t chunks = (R + kPrepChunk - 1) / kPrepChunk;
  const int P = chunks < kPrepMax ? (int)chunks : kPrepMax;
  hipLaunchKernelGGL(dedup_prep_kernel, dim3(P), dim3(kRadixThreads), 0, st, keys, Ri, w);
  int64_t rounds = (R + kAggRound - 1) / kAggRound;
  if (rounds > 4096) rounds = 4096;
  hipLaunchKernelGGL(dense_mark_kernel, dim3((unsigned)rounds), dim3(kRadixThreads), 0, st, Ri,
                     P, w);
  hipLaunchKernelGGL(dense_groups_kernel, dim3((unsigned)nvb), dim3(kRadixThreads), 0, st, Ri,
                     w, uk, fi, cnt, nu);
  int64_t ib = (R + 255) / 256;
  if (ib > 8192) ib = 8192;
  hipLaunchKernelGGL(dense_inverse_kernel, dim3((unsigned)ib), dim3(256), 0, st, Ri, w, inv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int G = nb < kRadixGridMax ? nb : kRadixGridMax;
  if (G > capacity) G = capacity;
  // an ordinary launch: G is at most what the device holds at once, so every
  // workgroup becomes resident (a cooperative launch would only add ~17 us of
  // set-up to every call, the dense path's included)
  hipLaunchKernelGGL(radix_sort_kernel, dim3(G), dim3(kRadixThreads), 0, st, Ri, nb, w, uk, fi,
                     cnt, inv, nu);
  return hipGetLastError();
}

}  // namespace hs
