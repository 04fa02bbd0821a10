// Reuse-driven priorities of the fused nodes and the ready-set order.
//
// HeraSys Eq. 3: a fused node v* contributes the sum of the contributions
// phi_v of all the logical nodes merged into it, so a node shared by many
// queries ranks higher.  Eq. 7 (also Algorithm 1, phase 2): the priority of a
// ready node is pi = alpha / (S_q + eps) + gamma * phi + delta * y, with S_q
// the remaining-time estimate of the node's query and y its heavy-node flag;
// the ready queues are ordered by pi, descending.
//
// Per fused node g (a group of hs_dedup):
//   phi*_g = sum over requests i with inverse[i] = g of phi_i, where each
//            phi_i (fp32, clamped to [0, 2^16), NaN as 0) is first truncated
//            to a multiple of 2^-24; the sum is exact (64-bit integer
//            atomics in units of 2^-24, so the order of the additions does
//            not matter) and rounded once to fp64;
//   pi_g   = ((alpha / (S_s + eps)) + gamma * phi*_g) + delta * y_s in fp64,
//            each operation rounded to nearest (no fused multiply-add), for
//            the surviving request s = first_index[g] (the node the merged
//            ones are redirected to);
//   order  = the fused nodes sorted by pi descending, then by g ascending
//            (-0 counts as +0).
// Both sides of a comparison therefore compute the same bits.
//
// Sort: chunks of kSortChunk (key, g) pairs are sorted in LDS by a bitonic
// network, then merged pairwise: each element's place in the merged run is
// its place in its own run plus the number of keys of the sibling run below
// it (binary search; keys are unique).  The number of merge passes follows
// the plan's distinct-key capacity, and a pass over runs wider than n_u is a
// plain copy, so the result always ends in the same buffer.
#include "common.h"

namespace hs {

constexpr int kPrioThreads = 256;
constexpr int kSmallMax = 4096;      // fused nodes handled by one workgroup
constexpr int kSmallThreads = 1024;
constexpr int kSortChunk = 1024;     // items per chunk of the many-node sort
constexpr int kSortThreads = 512;
constexpr double kPhiUnit = 16777216.0;   // 2^24 units per 1.0

struct SortItem {
  uint64_t key;   // ~(ordered bits of pi): ascending key = descending pi
  uint32_t g;
  uint32_t pad;
};

__device__ __forceinline__ bool item_less(const SortItem &a, const SortItem &b) {
  return a.key < b.key || (a.key == b.key && a.g < b.g);
}

// phi_i in units of 2^-24 (clamped to [0, 2^16), NaN as 0; < 2^40)
__device__ __forceinline__ uint64_t phi_units(float f) {
  f = f > 0.0f ? f : 0.0f;                         // negative and NaN -> 0
  f = f < 65536.0f ? f : 65535.99609375f;          // largest fp32 below 2^16
  // f * 2^24 is exact in fp32; truncation gives the units
  return (uint64_t)__float2ll_rz(f * 16777216.0f);
}

// phi* and pi of fused node g from its unit sum, and its sort item.
__device__ __forceinline__ SortItem node_priority(uint64_t units, int64_t g,
                                                  const int32_t *__restrict__ first_index,
                                                  const float *__restrict__ s_hat,
                                                  const uint8_t *__restrict__ heavy, int64_t R,
                                                  double alpha, double gamma, double delta,
                                                  double eps, double *__restrict__ phi_out,
                                                  double *__restrict__ pi_out) {
  // units < 2^63: one correctly rounded conversion, then an exact scaling
  const double ph = __dmul_rn(__ll2double_rn((long long)units), 1.0 / kPhiUnit);
  const int64_t s = first_index[g];
  const bool ok = s >= 0 && s < R;
  const double sq = ok ? (double)s_hat[s] : 0.0;
  const double y = ok && heavy ? (heavy[s] ? 1.0 : 0.0) : 0.0;
  double p = __dadd_rn(__ddiv_rn(alpha, __dadd_rn(sq, eps)), __dmul_rn(gamma, ph));
  p = __dadd_rn(p, __dmul_rn(delta, y));
  p = p == 0.0 ? 0.0 : p;   // -0 -> +0
  if (phi_out) phi_out[g] = ph;
  if (pi_out) pi_out[g] = p;
  const uint64_t b = (uint64_t)__double_as_longlong(p);
  const uint64_t ord = (b >> 63) ? ~b : (b | 0x8000000000000000ull);   // ascending with pi
  SortItem it;
  it.key = ~ord;
  it.g = (uint32_t)g;
  it.pad = 0u;
  return it;
}

// In-place ascending bitonic sort of sh[0, p2) (p2 a power of two, padded).
// Pair i of a stage joins items lo = 2i - (i mod stride) and lo + stride; a
// wave takes pairs [64 w, 64 w + 64) (and the same range one workgroup size
// further on, and so on), whose items lie in its own 128-item blocks
// whenever stride <= 64.  Such
// stages only need the wave's own LDS accesses ordered (a wavefront fence);
// a workgroup barrier follows the stages with larger strides and the last
// stage of each size.
__device__ __forceinline__ void bitonic_lds(SortItem *sh, int p2) {
  const int tid = threadIdx.x;
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < p2 / 2; i += blockDim.x) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const SortItem a = sh[lo], b = sh[hi];
        if (item_less(b, a) == up) {
          sh[lo] = b;
          sh[hi] = a;
        }
      }
      if (stride > 64 || stride == 1) {
        __syncthreads();
      } else {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
  }
}
static_assert(kSortThreads % 64 == 0 && kSmallThreads % 64 == 0, "whole waves");

__device__ __forceinline__ SortItem pad_item() {
  SortItem pad;
  pad.key = ~0ull;
  pad.g = 0xffffffffu;
  pad.pad = 0u;
  return pad;
}

// The whole step in one workgroup when at most kSmallMax fused nodes are
// possible: unit sums in LDS (64-bit LDS atomics), priorities, sort, order.
__global__ __launch_bounds__(kSmallThreads) void priority_small_kernel(
    const int32_t *__restrict__ inverse, const float *__restrict__ phi,
    const int32_t *__restrict__ first_index, const float *__restrict__ s_hat,
    const uint8_t *__restrict__ heavy, int64_t R, int64_t n_unique,
    const int64_t *__restrict__ nu_dev, int64_t cap, double alpha, double gamma, double delta,
    double eps, double *__restrict__ phi_out, double *__restrict__ pi_out,
    int32_t *__restrict__ order) {
  __shared__ unsigned long long units[kSmallMax];
  __shared__ SortItem sh[kSmallMax];
  const int64_t nu = read_nu(n_unique, nu_dev, cap);   // <= cap <= kSmallMax
  const int tid = threadIdx.x;
  for (int g = tid; g < nu; g += kSmallThreads) units[g] = 0ull;
  __syncthreads();
  for (int64_t i = tid; i < R; i += kSmallThreads) {
    const int32_t g = inverse[i];
    if (g < 0 || g >= nu) continue;
    const uint64_t u = phi_units(phi[i]);
    if (u) atomicAdd(&units[g], (unsigned long long)u);
  }
  __syncthreads();
  int p2 = 1;
  while (p2 < nu) p2 <<= 1;
  for (int g = tid; g < p2; g += kSmallThreads)
    sh[g] = g < nu ? node_priority(units[g], g, first_index, s_hat, heavy, R, alpha, gamma,
                                   delta, eps, phi_out, pi_out)
                   : pad_item();
  __syncthreads();
  bitonic_lds(sh, p2);
  for (int g = tid; g < nu; g += kSmallThreads) order[g] = (int32_t)sh[g].g;
}

// Unit sums for many requests: each workgroup adds up rounds of
// kAggRound consecutive requests in an LDS table keyed by fused node (hot
// nodes of a Zipf mix appear many times per round), then adds each entry to
// the global sums with one atomic.
constexpr int kAggRound = 1024, kAggSlots = 2048;
__global__ __launch_bounds__(kPrioThreads) void priority_sum_agg_kernel(
    const int32_t *__restrict__ inverse, const float *__restrict__ phi, int64_t R,
    int64_t n_unique, const int64_t *__restrict__ nu_dev, int64_t cap,
    uint64_t *__restrict__ units) {
  __shared__ int32_t tkey[kAggSlots];
  __shared__ unsigned long long tval[kAggSlots];
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int tid = threadIdx.x;
  for (int64_t r0 = (int64_t)blockIdx.x * kAggRound; r0 < R;
       r0 += (int64_t)gridDim.x * kAggRound) {
    for (int j = tid; j < kAggSlots; j += kPrioThreads) {
      tkey[j] = -1;
      tval[j] = 0ull;
    }
    __syncthreads();
    for (int j = tid; j < kAggRound; j += kPrioThreads) {
      const int64_t i = r0 + j;
      if (i >= R) break;
      const int32_t g = inverse[i];
      if (g < 0 || g >= nu) continue;
      const uint64_t u = phi_units(phi[i]);
      if (!u) continue;
      // open addressing; at most kAggRound keys in kAggSlots slots
      uint32_t h = ((uint32_t)g * 2654435761u) & (kAggSlots - 1);
      for (;;) {
        const int32_t prev = atomicCAS(&tkey[h], -1, g);
        if (prev == -1 || prev == g) break;
        h = (h + 1) & (kAggSlots - 1);
      }
      atomicAdd(&tval[h], (unsigned long long)u);
    }
    __syncthreads();
    for (int j = tid; j < kAggSlots; j += kPrioThreads)
      if (tkey[j] >= 0 && tval[j])
        atomicAdd((unsigned long long *)&units[tkey[j]], tval[j]);
    __syncthreads();
  }
}

__global__ void priority_clear_kernel(uint64_t *__restrict__ units, int64_t n_unique,
                                      const int64_t *__restrict__ nu_dev, int64_t cap) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nu;
       g += (int64_t)gridDim.x * blockDim.x)
    units[g] = 0ull;
}

__global__ void priority_pi_kernel(const uint64_t *__restrict__ units,
                                   const int32_t *__restrict__ first_index,
                                   const float *__restrict__ s_hat,
                                   const uint8_t *__restrict__ heavy, int64_t R,
                                   int64_t n_unique, const int64_t *__restrict__ nu_dev,
                                   int64_t cap, double alpha, double gamma, double delta,
                                   double eps, double *__restrict__ phi_out,
                                   double *__restrict__ pi_out, SortItem *__restrict__ items) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nu;
       g += (int64_t)gridDim.x * blockDim.x)
    items[g] = node_priority(units[g], g, first_index, s_hat, heavy, R, alpha, gamma, delta, eps,
                             phi_out, pi_out);
}

// Bitonic sort of each kSortChunk-item chunk of the first n_u items.
__global__ __launch_bounds__(kSortThreads) void priority_chunk_sort_kernel(
    SortItem *__restrict__ items, int64_t n_unique, const int64_t *__restrict__ nu_dev,
    int64_t cap) {
  __shared__ SortItem sh[kSortChunk];
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int64_t c0 = (int64_t)blockIdx.x * kSortChunk;
  if (c0 >= nu) return;
  const int n = (int)(nu - c0 < kSortChunk ? nu - c0 : kSortChunk);
  int p2 = 1;
  while (p2 < n) p2 <<= 1;
  const int tid = threadIdx.x;
  for (int i = tid; i < p2; i += kSortThreads) sh[i] = i < n ? items[c0 + i] : pad_item();
  __syncthreads();
  bitonic_lds(sh, p2);
  for (int i = tid; i < n; i += kSortThreads) items[c0 + i] = sh[i];
}

// Merge pass: runs of `width` sorted items in src -> runs of 2 * width in dst.
__global__ void priority_merge_kernel(const SortItem *__restrict__ src,
                                      SortItem *__restrict__ dst, int64_t width,
                                      int64_t n_unique, const int64_t *__restrict__ nu_dev,
                                      int64_t cap) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < nu;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int64_t a0 = p / (2 * width) * (2 * width);
    const int64_t b0 = a0 + width;
    const SortItem x = src[p];
    if (b0 >= nu) {   // no sibling run: copy
      dst[p] = x;
      continue;
    }
    const bool in_a = p < b0;
    // sibling run [o0, o1)
    const int64_t o0 = in_a ? b0 : a0;
    const int64_t o1 = in_a ? (b0 + width < nu ? b0 + width : nu) : b0;
    int64_t lo = o0, hi = o1;   // first sibling item not below x
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (item_less(src[mid], x)) lo = mid + 1;
      else hi = mid;
    }
    const int64_t own = in_a ? p - a0 : p - b0;
    dst[a0 + own + (lo - o0)] = x;
  }
}

__global__ void priority_order_kernel(const SortItem *__restrict__ items, int64_t n_unique,
                                      const int64_t *__restrict__ nu_dev, int64_t cap,
                                      int32_t *__restrict__ order) {
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < nu;
       p += (int64_t)gridDim.x * blockDim.x)
    order[p] = (int32_t)items[p].g;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t priority_workspace_bytes(int64_t cap) {
  const size_t c = (size_t)(cap > 0 ? cap : 1);
  return align256(c * 8) + 2 * align256(c * sizeof(SortItem));
}

static unsigned grid_of(int64_t n, int threads) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 4096) b = 4096;
  return (unsigned)b;
}

hipError_t launch_priority(const int32_t *inverse, const int32_t *first_index, int64_t R,
                           int64_t n_unique, const int64_t *nu_dev, int64_t cap,
                           const float *phi, const float *s_hat, const uint8_t *heavy,
                           double alpha, double gamma, double delta, double eps, double *phi_out,
                           double *pi_out, int32_t *order, void *ws, hipStream_t st) {
  const int64_t n = n_unique >= 0 ? n_unique : cap;   // launch bound
  if (cap <= kSmallMax) {
    hipLaunchKernelGGL(priority_small_kernel, dim3(1), dim3(kSmallThreads), 0, st, inverse, phi,
                       first_index, s_hat, heavy, R, n_unique, nu_dev, cap, alpha, gamma, delta,
                       eps, phi_out, pi_out, order);
    return hipGetLastError();
  }
  unsigned char *base = (unsigned char *)ws;
  uint64_t *units = (uint64_t *)base;
  SortItem *buf0 = (SortItem *)(base + align256((size_t)(cap > 0 ? cap : 1) * 8));
  SortItem *buf1 = buf0 + align256((size_t)(cap > 0 ? cap : 1) * sizeof(SortItem)) /
                              sizeof(SortItem);
  hipLaunchKernelGGL(priority_clear_kernel, dim3(grid_of(n, kPrioThreads)), dim3(kPrioThreads),
                     0, st, units, n_unique, nu_dev, cap);
  hipLaunchKernelGGL(priority_sum_agg_kernel, dim3(grid_of(R, kAggRound)), dim3(kPrioThreads), 0,
                     st, inverse, phi, R, n_unique, nu_dev, cap, units);
  hipLaunchKernelGGL(priority_pi_kernel, dim3(grid_of(n, kPrioThreads)), dim3(kPrioThreads), 0,
                     st, units, first_index, s_hat, heavy, R, n_unique, nu_dev, cap, alpha, gamma,
                     delta, eps, phi_out, pi_out, buf0);
  const int64_t chunks = (n + kSortChunk - 1) / kSortChunk;
  hipLaunchKernelGGL(priority_chunk_sort_kernel, dim3((unsigned)(chunks > 0 ? chunks : 1)),
                     dim3(kSortThreads), 0, st, buf0, n_unique, nu_dev, cap);
  SortItem *src = buf0, *dst = buf1;
  for (int64_t w = kSortChunk; w < n; w *= 2) {
    hipLaunchKernelGGL(priority_merge_kernel, dim3(grid_of(n, kPrioThreads)), dim3(kPrioThreads),
                       0, st, src, dst, w, n_unique, nu_dev, cap);
    SortItem *t = src;
    src = dst;
    dst = t;
  }
  hipLaunchKernelGGL(priority_order_kernel, dim3(grid_of(n, kPrioThreads)), dim3(kPrioThreads),
                     0, st, src, n_unique, nu_dev, cap, order);
  return hipGetLastError();
}

}  // namespace hs
