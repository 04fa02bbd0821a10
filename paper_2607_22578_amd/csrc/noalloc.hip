// Scratch memory for the entry point that allocates nothing
// (hs_score_topk_noalloc): a file-scope device array, one instance per GPU,
// held by the library until the process ends.  Host code never uses the
// array's name as an address: at a device's first use the device address is
// taken once with hipGetSymbolAddress (that device current) and kept per
// device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.h"

namespace hs {

constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;   // 64 MiB per GPU
static_assert(kNoAllocScratchBytes % 256 == 0, "scratch keeps 256-byte alignment");

__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

// Device address of the current device's scratch array (set up on the first
// call for that device).  Returns hipSuccess and *ptr, or the HIP error.
hipError_t noalloc_scratch(void **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p % 256) != 0) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace hs
