// ccq_util.hip -- small device utilities of the C ABI.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// dst[i] = src ? src[i] : 0 (a kernel rather than a memset/memcpy node, so the
// call stays safe to capture in a HIP graph).
__global__ void copy_or_zero_kernel(float* dst, const float* src, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src ? src[i] : 0.f;
}

hipError_t launch_copy_or_zero(float* dst, const float* src, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(copy_or_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, dst, src, n);
  return hipGetLastError();
}

}  // namespace ccq
