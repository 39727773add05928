// Fixed device workspace for the entry point that allocates nothing
// (aires_spgemm_noalloc): one file-scope array per device, living until the
// process ends.  Host code never uses the array's name as an address (in
// host code it is only a stand-in for the symbol); it asks the runtime for
// the array's device address once per device, with that device current,
// and passes that address to kernels and copies.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "scratch.h"

namespace {

// every call on a device shares this array; see aires_spgemm_noalloc
static __device__ __align__(256) unsigned char scratch[aires::kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

namespace aires {

hipError_t scratch_address(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace aires
