// Static scratch array of as2d_verify_static (include/as2d.h): the pass
// buffers of a verification call whose caller cannot allocate device
// memory (code under graph capture, tight serving loops) live here instead
// of in memory the library allocates.
//
// The array is a device global: each GPU the library runs on holds its own
// copy, at its own address, until the process ends.  In host code its name
// is only a host-side stand-in; the device address is looked up once per
// device (with that device current) and used for every kernel argument and
// copy.  Every call on one GPU shares the array and finds the previous
// call's contents in it; calls that overlap on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace as2d {

constexpr size_t kStaticScratchBytes = 32ull << 20;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices] = {};
std::mutex g_scratch_mu;
}  // namespace

hipError_t static_scratch(void** ptr, size_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

}  // namespace as2d
