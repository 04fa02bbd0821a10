// Shared device/host definitions of libhsmerge (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/hs_merge.h"

namespace hs {

constexpr int kWave = 64;

// ---- ordered 64-bit result keys --------------------------------------------
// A (score, row) pair packs into one uint64 whose unsigned order is the result
// order: higher score first, then lower row.  The high word maps the fp32 bit
// pattern to an order-preserving unsigned integer (with -0.0 folded onto +0.0
// so that both compare equal); the low word is ~row.  Key 0 is the empty slot
// (it sorts below every real key) and decodes to (-inf, -1).

__device__ __forceinline__ uint32_t ord_score(float s) {
  uint32_t b = __float_as_uint(s);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float unord_score(uint32_t o) {
  uint32_t b = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(b);
}

__device__ __forceinline__ uint64_t make_key(float s, uint32_t row) {
  return ((uint64_t)ord_score(s) << 32) | (uint64_t)(~row);
}

__device__ __forceinline__ void decode_key(uint64_t key, float &s, int32_t &row) {
  if (key == 0ull) {
    s = -__builtin_inff();
    row = -1;
  } else {
    s = unord_score((uint32_t)(key >> 32));
    row = (int32_t)(~(uint32_t)key);
  }
}

// ---- work split shared by the partial-score and merge kernels -------------
// Both kernels derive the same decomposition from (n_unique, N, grid size):
// queries in tiles of mq, corpus in tiles of nc, and S slices of the corpus per
// query tile; a work item is (query tile, slice).  S is picked among the
// values that make qtiles * S about r whole rounds of the persistent grid
// (r = 1..8) as the one with the least per-workgroup work,
// rounds * ceil(ntiles / S); S never exceeds smax (the merge bound S*k) nor the
// number of corpus tiles.
struct Split {
  int64_t nu;      // distinct queries
  int64_t qtiles;  // ceil(nu / mq)
  int64_t ntiles;  // ceil(N / nc)
  int64_t S;       // corpus slices per query tile
};

__host__ __device__ __forceinline__ Split make_split(int64_t nu, int64_t N, int mq, int nc,
                                                     int64_t grid, int64_t smax) {
  Split sp;
  sp.nu = nu;
  sp.qtiles = (nu + mq - 1) / mq;
  sp.ntiles = (N + nc - 1) / nc;
  sp.S = 1;
  if (sp.qtiles <= 0 || sp.ntiles <= 0 || grid <= 0) return sp;
  uint32_t cap = (uint32_t)(smax < sp.ntiles ? smax : sp.ntiles);
  if (cap < 1) cap = 1;
  const uint32_t qt = (uint32_t)sp.qtiles, nt = (uint32_t)sp.ntiles, gr = (uint32_t)grid;
  uint64_t best_cost = ~0ull;
  uint32_t best = 1;
  for (uint32_t r = 1; r <= 8; ++r) {
    uint32_t s = (uint32_t)(((uint64_t)r * gr) / qt);
    if (s < 1) s = 1;
    if (s > cap) s = cap;
    const uint64_t items = (uint64_t)qt * s;
    const uint64_t cost = ((items + gr - 1) / gr) * (uint64_t)((nt + s - 1) / s);
    if (cost < best_cost || (cost == best_cost && s < best)) {
      best_cost = cost;
      best = s;
    }
  }
  sp.S = best;
  return sp;
}

// Logical id of this workgroup: consecutive ids on one XCD (workgroups are
// dispatched round-robin over the 8 XCDs; grid is a multiple of 8).
__device__ __forceinline__ int logical_wg(int grid) {
  int b = blockIdx.x;
  return (b & 7) * (grid >> 3) + (b >> 3);
}

__device__ __forceinline__ int64_t read_nu(int64_t n_unique, const int64_t *n_unique_dev,
                                           int64_t cap) {
  int64_t nu = n_unique >= 0 ? n_unique : *n_unique_dev;
  if (nu < 0) nu = 0;
  if (nu > cap) nu = cap;
  return nu;
}

}  // namespace hs
