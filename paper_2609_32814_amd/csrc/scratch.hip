// The library's one static device buffer: the workspace of
// star_decode_noalloc, for callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  Each device that runs the library holds its own copy of the
// array until the process ends.
//
// In host code the array's name is only a host-side stand-in for the
// symbol, not a device address: the device address is taken once per device
// with hipGetSymbolAddress (with that device current) and kept, and only
// that address is ever handed to kernels or fill launches.
#include <atomic>

#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace starq {

namespace {

__device__ __attribute__((aligned(256))) unsigned char scratch[kDecodeScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

}  // namespace

hipError_t decode_scratch(void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    // first call on this device (it is current): look the symbol up.  Two
    // threads racing here both get the same address.
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_addr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace starq
