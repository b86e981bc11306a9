// Fixed per-device scratch array for steel_attn_fwd_noalloc: the live-block
// index of a fused call placed in a file-scope device array instead of
// memory the library allocates, for callers that cannot allocate.
//
// The array's name is a host-side stand-in in host code, not a device
// address: each device holds its own copy, whose address is looked up once
// per device (hipGetSymbolAddress, with that device current) and kept; only
// that address is ever handed to a kernel.
#include <mutex>

#include "internal.h"

namespace steel {

namespace {

__device__ __align__(256) char scratch[kNoAllocBytes];

constexpr int kMaxDev = 64;
std::mutex g_mu;
char* g_ptr[kMaxDev] = {};

}  // namespace

hipError_t noalloc_scratch(int dev, char** ptr) {
  *ptr = nullptr;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_ptr[dev]) {
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e != hipSuccess) return e;
    if (prev != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev != dev) (void)hipSetDevice(prev);
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255u) != 0) return hipErrorInvalidSymbol;
    g_ptr[dev] = static_cast<char*>(p);
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace steel
