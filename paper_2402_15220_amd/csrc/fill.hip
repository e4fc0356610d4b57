// Device-side fill for library-owned buffers. Used instead of
// hipMemsetAsync on the caller's stream, so that a caller who captures
// library calls into a HIP graph records a kernel node rather than a memset
// node.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "kernels.hpp"

namespace ca {
namespace {

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n,
                                                       int32_t value) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i] = value;
}

}  // namespace

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t value, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (!p) return hipErrorInvalidValue;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 1024);
  fill_i32_kernel<<<static_cast<unsigned>(blocks), 256, 0, stream>>>(p, n, value);
  return hipGetLastError();
}

}  // namespace ca
