// Static scratch memory of the allocation-free forward (ga_forward_noalloc).
//
// The forward's device scratch (groups, centroids, representatives, the
// grouping kernel's moved-key records and barrier words, the attention's
// value means) lives in one file-scope device array.  Each GPU the library
// runs on holds its own copy of the array, at its own address, until the
// process ends.  In host code the array's name is only a host-side stand-in:
// its device address is looked up once per device with hipGetSymbolAddress
// (with that device current) and only that address is handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ga_internal.h"

namespace ga {
namespace {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device, null until looked up

}  // namespace

hipError_t static_scratch(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255u) != 0) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace ga
