// Device scratch of the allocation-free attention entry point
// (ca_attention_noalloc): one statically sized array in the code object, so
// every GPU the library is loaded on holds its own copy from module load
// until the process ends, and using it needs no allocation.
//
// In host code the array's name is only a host-side stand-in for the symbol,
// not a device address: passing it to a kernel would fault. The address of
// each device's copy is taken once per device, with that device current,
// through hipGetSymbolAddress, and only that address is used afterwards.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.hpp"

static __device__ __align__(256) char scratch[ca::kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
char* g_addr[kMaxDevices] = {};

}  // namespace

namespace ca {

hipError_t scratch_address(char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_addr[dev] = static_cast<char*>(p);
  }
  *out = g_addr[dev];
  return hipSuccess;
}

}  // namespace ca
