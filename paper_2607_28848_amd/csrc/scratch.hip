// scratch.hip -- device scratch of the allocation-free forward entry point
// (dsv_cobatch_fwd_noalloc): a fixed array in the library's own device memory
// that stands in for the caller's workspace.
//
// The array's name is a host-side stand-in, not a device address.  Each
// device holds its own copy at its own address, so the address is looked up
// once per device (with that device current) and kept; kernels and copies take
// that address, never the array's name.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

static __device__ __align__(256) char scratch[dsv::kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

namespace dsv {

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr || (reinterpret_cast<uintptr_t>(p) & 255) != 0) return hipErrorInvalidValue;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace dsv
