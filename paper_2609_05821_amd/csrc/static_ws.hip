// Fixed device scratch of the allocation-free scoring entry point
// (conduit_score_noalloc).  The array lives in the library's code object, so
// every GPU the library is loaded on holds its own copy, at its own address,
// until the process ends.  Host code never passes the array's name to a
// kernel or a copy (in host code it is a host-side stand-in, not a device
// address): it resolves the device address once per device with
// hipGetSymbolAddress and uses that pointer.
#include <mutex>

#include "common.h"

namespace {

__device__ __align__(256) unsigned char scratch[conduit::kStaticScoreScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

}  // namespace

namespace conduit {

hipError_t static_score_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255u)) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace conduit
