// Library-owned device scratch for the entry point that allocates nothing
// (moeca_forward_noalloc).
//
// One file-scope device array per GPU, kScratchBytes long, loaded with the
// code object and held until the process ends.  Host code never passes the
// array's name to a kernel (in host code the name is a stand-in, not a
// device address): its device address is looked up once per device with
// hipGetSymbolAddress, with that device current, and that address is what
// the launches receive.  Every call on a GPU shares that GPU's array, so
// calls that overlap on one GPU race; each call writes every byte it later
// reads, so nothing has to be cleared between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[moeca::kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

namespace moeca {

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255u) != 0) return hipErrorInvalidSymbol;
    g_addr[dev] = p;
  }
  *out = g_addr[dev];
  return hipSuccess;
}

}  // namespace moeca
