// Scratch memory of xattn_forward_noalloc: a file-scope device array that the
// library owns, so that the forward pass runs without any allocation. Each
// GPU the library runs on holds its own copy of the array (in the code
// object loaded on that device) until the process ends.
//
// In host code the name `scratch` is a host-side stand-in, not a device
// address: the array's device address is fetched once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.h"

namespace {

__device__ __attribute__((aligned(256))) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];  // device address of `scratch` per device, guarded by g_mu

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}
