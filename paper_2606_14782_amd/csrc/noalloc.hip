// Static device scratch of the allocation-free entry point
// (bacon_window_lse_static): a file-scope device array, one copy per GPU the
// library runs on, held until the process ends.  Host code never uses the
// array's name as an address: the first call on a device looks its address
// up there (hipGetSymbolAddress, with that device current) and keeps it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace bacon {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(void **ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace bacon
