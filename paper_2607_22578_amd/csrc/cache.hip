// Cross-window result reuse: a device-resident result store keyed by
// signature.
//
// HeraSys Sec. 3.3 (II), asynchronous cache reuse: a node that arrives after
// its window has closed, and whose signature matches an already completed
// node, takes that node's result instead of running again.  Here a window's
// distinct keys (after the dedup of step 1) are looked up in a store that
// previous windows filled; hits receive the stored top-k rows, only the
// misses are scored, and their results are stored for later windows.
//
// The store is direct-mapped: key -> slot by Fibonacci hashing (the key
// times 2^64 / golden ratio, top log2(C) bits), one result per slot.  A hit
// needs the slot to be valid and to hold the same key.  When several misses
// of one window map to the same slot, the one with the largest distinct-key
// position (the largest key, since distinct keys are ascending) is stored;
// a store replaces whatever the slot held before.  So the store's content
// after every window is a function of the windows alone, whatever the launch
// order of the threads.
//
// Layout of the caller's buffer (each array 256-byte aligned): keys [C]
// int64 | valid [C] int32 | claim [C] int32 | score [C x k] fp32 |
// index [C x k] int32.
#include "common.h"

namespace hs {

struct CacheView {
  int64_t *keys;
  int32_t *valid;
  int32_t *claim;
  float *score;
  int32_t *index;
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t cache_layout(int64_t C, int k, void *base, CacheView *v) {
  unsigned char *p = (unsigned char *)base;
  size_t off = 0;
  CacheView w;
  w.keys = (int64_t *)(p + off);
  off += align256((size_t)C * 8);
  w.valid = (int32_t *)(p + off);
  off += align256((size_t)C * 4);
  w.claim = (int32_t *)(p + off);
  off += align256((size_t)C * 4);
  w.score = (float *)(p + off);
  off += align256((size_t)C * k * 4);
  w.index = (int32_t *)(p + off);
  off += align256((size_t)C * k * 4);
  if (v) *v = w;
  return off;
}

__device__ __forceinline__ uint32_t cache_slot(int64_t key, int bits) {
  const uint64_t h = (uint64_t)key * 0x9E3779B97F4A7C15ull;
  return bits > 0 ? (uint32_t)(h >> (64 - bits)) : 0u;
}

__global__ void cache_reset_kernel(CacheView v, int64_t C) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < C;
       i += (int64_t)gridDim.x * blockDim.x) {
    v.valid[i] = 0;
    v.claim[i] = -1;
  }
}

// Hit test and miss list, one workgroup: distinct keys in chunks of
// kCacheThreads, misses numbered in ascending key order by a block scan.
constexpr int kCacheThreads = 1024;

__global__ __launch_bounds__(kCacheThreads) void cache_lookup_kernel(
    CacheView v, int bits, const int64_t *__restrict__ uk, const int32_t *__restrict__ fi,
    int64_t n_unique, const int64_t *__restrict__ nu_dev, int64_t cap,
    int32_t *__restrict__ miss_pos, int32_t *__restrict__ miss_first,
    int64_t *__restrict__ n_miss) {
  __shared__ int32_t wsum[kCacheThreads / kWave + 1];
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  int64_t base = 0;
  for (int64_t u0 = 0; u0 < nu; u0 += kCacheThreads) {
    const int64_t u = u0 + tid;
    bool miss = false;
    uint32_t slot = 0;
    if (u < nu) {
      const int64_t key = uk[u];
      slot = cache_slot(key, bits);
      miss = !(v.valid[slot] != 0 && v.keys[slot] == key);
    }
    const uint64_t m = __builtin_amdgcn_ballot_w64(miss);
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    if (tid == 0) {
      int32_t acc = 0;
      for (int i = 0; i < kCacheThreads / kWave; ++i) {
        const int32_t t = wsum[i];
        wsum[i] = acc;
        acc += t;
      }
      wsum[kCacheThreads / kWave] = acc;
    }
    __syncthreads();
    if (u < nu) {
      if (miss) {
        const int64_t pos = base + wsum[w] + __popcll(m & ((1ull << lane) - 1ull));
        miss_pos[u] = (int32_t)pos;
        miss_first[pos] = fi[u];
        v.claim[slot] = -1;   // every miss of this window rewrites the same value
      } else {
        miss_pos[u] = -1;
      }
    }
    base += wsum[kCacheThreads / kWave];
    __syncthreads();
  }
  if (tid == 0) *n_miss = base;
}

// Hit rows of the store -> the window's top-k rows (misses untouched).
__global__ void cache_copy_hits_kernel(CacheView v, int bits, int k, const int64_t *__restrict__ uk,
                                       int64_t n_unique, const int64_t *__restrict__ nu_dev,
                                       int64_t cap, const int32_t *__restrict__ miss_pos,
                                       float *__restrict__ out_s, int32_t *__restrict__ out_i) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int64_t total = nu * k;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t u = e / k;
    if (miss_pos[u] >= 0) continue;
    const int64_t src = (int64_t)cache_slot(uk[u], bits) * k + (e - u * k);
    out_s[e] = v.score[src];
    out_i[e] = v.index[src];
  }
}

// Insert, phase 1: every miss bids for its slot; the largest position wins.
__global__ void cache_claim_kernel(CacheView v, int bits, const int64_t *__restrict__ uk,
                                   int64_t n_unique, const int64_t *__restrict__ nu_dev,
                                   int64_t cap, const int32_t *__restrict__ miss_pos) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nu;
       u += (int64_t)gridDim.x * blockDim.x)
    if (miss_pos[u] >= 0) atomicMax(&v.claim[cache_slot(uk[u], bits)], (int32_t)u);
}

// Insert, phase 2: the winner of a slot stores its key and top-k row.
__global__ void cache_store_kernel(CacheView v, int bits, int k, const int64_t *__restrict__ uk,
                                   int64_t n_unique, const int64_t *__restrict__ nu_dev,
                                   int64_t cap, const int32_t *__restrict__ miss_pos,
                                   const float *__restrict__ top_s,
                                   const int32_t *__restrict__ top_i) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int64_t total = nu * k;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t u = e / k, j = e - u * k;
    if (miss_pos[u] < 0) continue;
    const int64_t key = uk[u];
    const uint32_t slot = cache_slot(key, bits);
    if (v.claim[slot] != (int32_t)u) continue;
    v.score[(int64_t)slot * k + j] = top_s[e];
    v.index[(int64_t)slot * k + j] = top_i[e];
    if (j == 0) {
      v.keys[slot] = key;
      v.valid[slot] = 1;
    }
  }
}

static int log2_exact(int64_t C) {
  int b = 0;
  while (((int64_t)1 << b) < C) ++b;
  return b;
}

static unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > 4096) b = 4096;
  return (unsigned)b;
}

hipError_t launch_cache_reset(void *cache, int64_t C, int k, hipStream_t st) {
  CacheView v;
  cache_layout(C, k, cache, &v);
  hipLaunchKernelGGL(cache_reset_kernel, dim3(grid_for(C)), dim3(256), 0, st, v, C);
  return hipGetLastError();
}

hipError_t launch_cache_lookup(void *cache, int64_t C, int k, const int64_t *uk,
                               const int32_t *fi, int64_t n_unique, const int64_t *nu_dev,
                               int64_t cap, float *out_s, int32_t *out_i, int32_t *miss_pos,
                               int32_t *miss_first, int64_t *n_miss, hipStream_t st) {
  CacheView v;
  cache_layout(C, k, cache, &v);
  const int bits = log2_exact(C);
  hipLaunchKernelGGL(cache_lookup_kernel, dim3(1), dim3(kCacheThreads), 0, st, v, bits, uk, fi,
                     n_unique, nu_dev, cap, miss_pos, miss_first, n_miss);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t worst = (n_unique >= 0 ? n_unique : cap) * k;
  hipLaunchKernelGGL(cache_copy_hits_kernel, dim3(grid_for(worst)), dim3(256), 0, st, v, bits, k,
                     uk, n_unique, nu_dev, cap, miss_pos, out_s, out_i);
  return hipGetLastError();
}

hipError_t launch_cache_insert(void *cache, int64_t C, int k, const int64_t *uk, int64_t n_unique,
                               const int64_t *nu_dev, int64_t cap, const int32_t *miss_pos,
                               const float *top_s, const int32_t *top_i, hipStream_t st) {
  CacheView v;
  cache_layout(C, k, cache, &v);
  const int bits = log2_exact(C);
  const int64_t n = n_unique >= 0 ? n_unique : cap;
  hipLaunchKernelGGL(cache_claim_kernel, dim3(grid_for(n)), dim3(256), 0, st, v, bits, uk,
                     n_unique, nu_dev, cap, miss_pos);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cache_store_kernel, dim3(grid_for(n * k)), dim3(256), 0, st, v, bits, k, uk,
                     n_unique, nu_dev, cap, miss_pos, top_s, top_i);
  return hipGetLastError();
}

}  // namespace hs
