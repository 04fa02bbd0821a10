// Host-only stand-ins for the device side of libhsmerge (the kernels and
// their launchers live in the .hip sources): used to build the C ABI's
// argument validation (api.cpp) with the host sanitizers, without a GPU.
// Each launcher only counts its calls; the workspace sizes follow simple
// formulas of the same shape as the real ones.
#include <hip/hip_runtime_api.h>

#include <cstddef>
#include <cstdint>

extern "C" {
int hs_stub_launches = 0;
}

namespace hs {
struct CacheView;
size_t dedup_workspace_bytes(int64_t R) { return R <= 4096 ? 0 : (size_t)R * 32; }
size_t score_workspace_bytes(int64_t cap, int64_t N, int64_t d, int k, int) {
  (void)N;
  (void)d;
  return ((size_t)cap * (size_t)k * 64 + 255) & ~(size_t)255;
}
size_t priority_workspace_bytes(int64_t cap) { return (size_t)cap * 16; }
size_t mfma_tiled_bytes(int64_t N, int64_t d, bool fp8) {
  return (size_t)((N + 383) / 384 * 384) * (size_t)((d + 63) / 64 * 64) * (fp8 ? 1u : 2u);
}
size_t cache_layout(int64_t C, int k, void *, CacheView *) {
  return ((size_t)C * (16 + 8 * (size_t)k) + 1023) & ~(size_t)255;
}
size_t noalloc_scratch_bytes() { return (size_t)64 << 20; }
hipError_t noalloc_scratch(void **ptr) {
  *ptr = nullptr;
  return hipErrorNoDevice;   // no GPU in a host-only build
}
#define HS_STUB(name, ...)          \
  hipError_t name(__VA_ARGS__) {    \
    ++hs_stub_launches;             \
    return hipSuccess;              \
  }
HS_STUB(launch_dedup, const int64_t *, int64_t, int64_t *, int32_t *, int32_t *, int32_t *,
        int64_t *, void *, hipStream_t)
HS_STUB(launch_gather, const void *, int64_t, int64_t, const void *, int, int64_t,
        const int64_t *, void *, hipStream_t)
HS_STUB(launch_deliver, const float *, const int32_t *, int64_t, const int32_t *, int64_t, int,
        float *, int32_t *, hipStream_t)
HS_STUB(launch_score_partial, const void *, const void *, const float *, int64_t, int64_t, int,
        int64_t, const int64_t *, int64_t, int, bool, void *, hipStream_t)
HS_STUB(launch_tile_corpus, const void *, int64_t, int64_t, bool, void *, hipStream_t)
HS_STUB(launch_topk_merge, const void *, int64_t, const int64_t *, int64_t, int64_t, int, int,
        float *, int32_t *, hipStream_t)
HS_STUB(launch_cache_reset, void *, int64_t, int, hipStream_t)
HS_STUB(launch_cache_lookup, void *, int64_t, int, const int64_t *, const int32_t *, int64_t,
        const int64_t *, int64_t, float *, int32_t *, int32_t *, int32_t *, int64_t *,
        hipStream_t)
HS_STUB(launch_cache_insert, void *, int64_t, int, const int64_t *, int64_t, const int64_t *,
        int64_t, const int32_t *, const float *, const int32_t *, hipStream_t)
HS_STUB(launch_signature, const uint32_t *, const uint8_t *, const int64_t *, int64_t,
        const uint8_t *, const int64_t *, int64_t, const int32_t *, const int32_t *, int64_t,
        int64_t, int64_t, int, uint8_t *, int64_t *, hipStream_t)
HS_STUB(launch_priority, const int32_t *, const int32_t *, int64_t, int64_t, const int64_t *,
        int64_t, const float *, const float *, const uint8_t *, double, double, double, double,
        double *, double *, int32_t *, void *, hipStream_t)
}  // namespace hs
