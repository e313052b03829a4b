// Library-owned scratch memory for lookme_inject_noalloc, the variant of
// lookme_inject that allocates nothing and needs no workspace (for callers
// that cannot allocate device memory, e.g. under stream capture).
//
// The array lives in this module's device data: every GPU the library runs
// on holds its own copy, at its own address, until the process ends.  Host
// code must never pass the array's name to a kernel (on the host it is only
// a stand-in symbol); its device address is looked up here once per device,
// with that device current, and kept.  Every call on one GPU shares that
// GPU's copy, so calls that overlap on one GPU (several streams, several
// host threads) race on it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace lookme {

static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_ptr[MAX_DEVICES] = {};
}  // namespace

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace lookme
