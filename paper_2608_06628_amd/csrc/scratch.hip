// scratch.hip -- the library-held scratch buffer of the entry points that
// allocate nothing (for callers that cannot call hipMalloc: code under graph
// capture, tight serving loops).
//
// The buffer is a file-scope device array; every GPU the library runs on
// holds its own copy, at its own address, until the process ends.  In host
// code the array's name is only a host-side stand-in, so its device address
// is looked up once per device (hipGetSymbolAddress, with that device
// current) and every kernel argument uses that address.  Calls that use the
// buffer on one GPU share it: calls that overlap in time on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "launch.h"

namespace hyb {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_device_ptr(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
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

}  // namespace hyb
