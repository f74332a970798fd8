// Device scratch of the no-allocation entry point (spec_verify_noalloc): a
// fixed array in the library's own device memory, which every GPU the
// library runs on holds until the process ends.  Host code never uses the
// array's name as an address: it takes each device's address of it once,
// with that device current, and passes that pointer to the kernels, exactly
// as it passes a caller's workspace to the other entry points.
#include <mutex>

#include "sv_internal.h"

namespace sv {
namespace {

static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDev = 64;
std::mutex g_mu;
void* g_ptr[kMaxDev];

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace sv
