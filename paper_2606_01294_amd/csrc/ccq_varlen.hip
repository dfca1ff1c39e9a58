// ccq_varlen.hip -- packed batches of sequences of different lengths.
//
// Sequence b of a packed batch holds rows cu[b] .. cu[b+1] - 1 of every
// [rows, H, d] tensor.  Every sequence is independent (its own states), so
// the packed batch is carried through the chunkwise path as a padded batch
// [B, T, H, d] (T the longest length): row t of sequence b is copied to
// padded row b T + t, and the rows past the sequence's end hold zeros.  A
// zero row leaves every state unchanged (k = v = 0 writes nothing; a zero
// log-gate or log-decay keeps S; beta = 0 makes the delta rule the identity)
// and, the path being causal, changes no output of the sequence's own rows.
// The only quantities the padding reaches are the running means of the
// contraction cache, Cbar_T = S^K / (t0 + T) and mu_T = m / (t0 + T), whose
// sums are unchanged but whose counts are not: varlen_cache_fix rescales
// them to the sequence's own count t0 + len_b.
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

// Cbar_T and mu_T of (sequence b, head h) = blockIdx.y: counts t0 + T ->
// t0 + len_b, blockIdx.x taking 256 of the head's dk * dk + dk values; a
// sequence with no tokens at all returns the initial cache.
__global__ void varlen_cache_fix_kernel(float* CT, float* muT, const float* C0, const float* mu0,
                                        const int* cu, int H, int dk, int T, long long t0) {
  const int bh = blockIdx.y, b = bh / H;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int nc = dk * dk;
  if (i >= nc + dk) return;
  const int len = seq_len(cu, b, T);
  const long long cnt = t0 + len;
  float* dst = i < nc ? (CT ? CT + (size_t)bh * nc + i : nullptr) : (muT ? muT + (size_t)bh * dk + (i - nc) : nullptr);
  if (!dst) return;
  if (cnt == 0) {
    const float* src = i < nc ? (C0 ? C0 + (size_t)bh * nc + i : nullptr) : (mu0 ? mu0 + (size_t)bh * dk + (i - nc) : nullptr);
    *dst = src ? *src : 0.f;
    return;
  }
  *dst *= (float)((double)(t0 + T) / (double)cnt);
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

hipError_t launch_varlen_cache_fix(float* CT, float* muT, const float* C0, const float* mu0, const int* cu,
                                   int B, int H, int dk, int T, long long t0, hipStream_t st) {
  if (B == 0 || H == 0 || (!CT && !muT)) return hipSuccess;
  const unsigned nx = (unsigned)((dk * dk + dk + 255) / 256);
  hipLaunchKernelGGL(varlen_cache_fix_kernel, dim3(nx, (unsigned)(B * H)), dim3(256), 0, st, CT, muT, C0, mu0, cu,
                     H, dk, T, t0);
  return hipGetLastError();
}

}  // namespace ccq
