// Steps 2 and 2': row gather dst[i] = src[index[i]]; step 5: delivery.
//
// HeraSys Sec. 3.3 (I): the surviving node runs once and its output flows to
// the downstream nodes of every related query.  Expressed as a gather (each
// destination row pulls from its source) the delivery has no write conflicts.
// The same kernel builds the representative query batch (index = survivor of
// each group) and the embedding rows of distinct chunk ids.
//
// A group of G threads copies one row with G consecutive vector accesses
// (16-byte when the row allows, else 4-byte), so a wavefront reads and writes
// whole contiguous row segments.  16-byte rows are stored nontemporally: the
// destination is not read again by the kernel, and streaming it past the
// caches leaves them to the source rows (~7% faster on 2 KiB rows).
#include "common.h"

namespace hs {

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
template <typename V>
__device__ __forceinline__ void copy_vec(const V *s, V *d) {
  *d = *s;
}
template <>
__device__ __forceinline__ void copy_vec<uint4>(const uint4 *s, uint4 *d) {
  __builtin_nontemporal_store(*(const u32x4_t *)s, (u32x4_t *)d);
}

template <typename V, typename I>
__global__ __launch_bounds__(256) void gather_rows_kernel(
    const V *__restrict__ src, int64_t src_rows, int vpr, int group, const I *__restrict__ index,
    int64_t n_out, const int64_t *__restrict__ n_out_dev, V *__restrict__ dst) {
  int64_t n = n_out;
  if (n_out_dev) {
    int64_t m = *n_out_dev;
    if (m < n) n = m;
  }
  const int rows_per_block = 256 / group;
  const int sub = threadIdx.x / group, lane = threadIdx.x % group;
  for (int64_t row = (int64_t)blockIdx.x * rows_per_block + sub; row < n;
       row += (int64_t)gridDim.x * rows_per_block) {
    int64_t r = (int64_t)index[row];
    if (r < 0 || r >= src_rows) continue;
    const V *s = src + r * vpr;
    V *d = dst + row * vpr;
    for (int c = lane; c < vpr; c += group) copy_vec(&s[c], &d[c]);
  }
}

template <typename V>
static hipError_t launch_gather_t(const void *src, int64_t src_rows, int64_t row_bytes,
                                  const void *index, int is64, int64_t n_out,
                                  const int64_t *n_out_dev, void *dst, hipStream_t st) {
  const int vpr = (int)(row_bytes / (int64_t)sizeof(V));
  int group = 1;
  while (group < vpr && group < 256) group <<= 1;
  const int rows_per_block = 256 / group;
  int64_t blocks = (n_out + rows_per_block - 1) / rows_per_block;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (is64)
    hipLaunchKernelGGL((gather_rows_kernel<V, int64_t>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const V *)src, src_rows, vpr, group, (const int64_t *)index, n_out,
                       n_out_dev, (V *)dst);
  else
    hipLaunchKernelGGL((gather_rows_kernel<V, int32_t>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const V *)src, src_rows, vpr, group, (const int32_t *)index, n_out,
                       n_out_dev, (V *)dst);
  return hipGetLastError();
}

hipError_t launch_gather(const void *src, int64_t src_rows, int64_t row_bytes, const void *index,
                         int is64, int64_t n_out, const int64_t *n_out_dev, void *dst,
                         hipStream_t st) {
  if (n_out <= 0) return hipSuccess;
  bool v16 = (row_bytes % 16 == 0) && (((uintptr_t)src | (uintptr_t)dst) % 16 == 0);
  if (v16)
    return launch_gather_t<uint4>(src, src_rows, row_bytes, index, is64, n_out, n_out_dev, dst,
                                  st);
  return launch_gather_t<uint32_t>(src, src_rows, row_bytes, index, is64, n_out, n_out_dev, dst,
                                   st);
}

// Step 5 in one launch: request i receives the k results of its group,
// out[i * k + j] = topk[inverse[i] * k + j] for scores and indices.  One
// thread per output element, so consecutive threads read and write
// consecutive elements of a row; groups outside [0, rows) are skipped.
__global__ __launch_bounds__(256) void deliver_kernel(const float *__restrict__ ts,
                                                      const int32_t *__restrict__ ti,
                                                      int64_t rows, const int32_t *__restrict__ inv,
                                                      int64_t R, int k, float *__restrict__ os,
                                                      int32_t *__restrict__ oi) {
  const int64_t total = R * k;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / k;
    const int64_t g = inv[i];
    if (g < 0 || g >= rows) continue;
    const int64_t src = g * k + (e - i * k);
    os[e] = ts[src];
    oi[e] = ti[src];
  }
}

hipError_t launch_deliver(const float *ts, const int32_t *ti, int64_t rows, const int32_t *inv,
                          int64_t R, int k, float *os, int32_t *oi, hipStream_t st) {
  const int64_t total = R * (int64_t)k;
  if (total <= 0) return hipSuccess;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(deliver_kernel, dim3((unsigned)blocks), dim3(256), 0, st, ts, ti, rows, inv,
                     R, k, os, oi);
  return hipGetLastError();
}

}  // namespace hs
