// ccq_varlen.hip -- padded copies of packed batches for the training step.
//
// Sequence b of a packed batch holds rows cu[b] .. cu[b+1] - 1 of every
// [rows, H, d] tensor.  The forward kernels read packed rows directly; the
// training step (ccq_fwd_bwd_varlen) runs on a padded batch [B, T, H, d] (T
// the longest length): row t of sequence b is copied to padded row b T + t
// and the rows past the sequence's end hold zeros.  A zero row leaves every
// state unchanged (k = v = 0 writes nothing; a zero log-gate or log-decay
// keeps S; beta = 0 makes the delta rule the identity) and, the path being
// causal, changes no output or gradient of the sequence's own rows; the
// training step returns no caches, so the padding's effect on the running
// means' counts does not arise.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

namespace {
// Length of sequence b, clamped to [0, T] (offsets are the caller's: a longer
// sequence is cut at T rather than read or written out of range).
__device__ __forceinline__ int seq_len(const int* cu, int b, int T) {
  const int n = cu[b + 1] - cu[b];
  return n < 0 ? 0 : (n > T ? T : n);
}

// Copy every unit of the padded rows of sequence blockIdx.y (grid-stride in
// x over T * units): TO_PADDED gathers (rows past the end zeroed), else
// scatters the sequence's rows back to the packed tensor.
template <typename V, bool TO_PADDED>
__global__ void varlen_copy_kernel(V* dst, const V* src, const int* cu, int T, long long units) {
  const int b = blockIdx.y;
  const int len = seq_len(cu, b, T);
  const long long packed0 = (long long)cu[b] * units, padded0 = (long long)b * T * units;
  const long long n = (long long)T * units;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x) {
    const bool live = i < (long long)len * units;
    if constexpr (TO_PADDED) {
      V x{};
      if (live) x = src[packed0 + i];
      dst[padded0 + i] = x;
    } else {
      if (live) dst[packed0 + i] = src[padded0 + i];
    }
  }
}

}  // namespace

hipError_t launch_varlen_copy(void* dst, const void* src, const int* cu, int B, int T, size_t row_bytes,
                              bool to_padded, hipStream_t st) {
  if (B == 0 || T == 0 || row_bytes == 0) return hipSuccess;
  if (row_bytes % 4 != 0) return hipErrorInvalidValue;
  const bool wide = row_bytes % 16 == 0;
  const long long units = (long long)(row_bytes / (wide ? 16 : 4));
  const long long n = (long long)T * units;
  long long bx = (n + 255) / 256;
  if (bx > 1024) bx = 1024;
  const dim3 grid((unsigned)bx, (unsigned)B);
  if (wide) {
    typedef uint4 V;
    if (to_padded)
      hipLaunchKernelGGL((varlen_copy_kernel<V, true>), grid, dim3(256), 0, st, static_cast<V*>(dst),
                         static_cast<const V*>(src), cu, T, units);
    else
      hipLaunchKernelGGL((varlen_copy_kernel<V, false>), grid, dim3(256), 0, st, static_cast<V*>(dst),
                         static_cast<const V*>(src), cu, T, units);
  } else {
    typedef uint32_t V;
    if (to_padded)
      hipLaunchKernelGGL((varlen_copy_kernel<V, true>), grid, dim3(256), 0, st, static_cast<V*>(dst),
                         static_cast<const V*>(src), cu, T, units);
    else
      hipLaunchKernelGGL((varlen_copy_kernel<V, false>), grid, dim3(256), 0, st, static_cast<V*>(dst),
                         static_cast<const V*>(src), cu, T, units);
  }
  return hipGetLastError();
}

}  // namespace ccq
