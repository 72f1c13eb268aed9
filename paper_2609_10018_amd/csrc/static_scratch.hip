// Activation scratch for callers that cannot allocate device memory (code
// under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
// one statically sized array per GPU, which the device code object holds
// from its load until the process ends.
//
// In host code the array's name is a host-side stand-in, not a device
// address.  Its device address is looked up once per device, with that
// device current, through hipGetSymbolAddress; every later use (kernel
// arguments, copies) takes that address.  Every caller on one GPU shares the
// array, which keeps the last call's contents: calls that overlap on one GPU
// (several streams, or several handles) race on it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kernels.h"

namespace elasto {
namespace {

__device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch(void** ptr, int64_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

}  // namespace elasto
