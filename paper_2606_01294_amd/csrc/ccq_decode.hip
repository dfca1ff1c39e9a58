// ccq_decode.hip -- one recurrent CCQ step per sequence (Alg. 2, recurrent
// inference) on the cache triple (S, Cbar, mu), updated in place.
//
// With t the 1-based position of the new token (t0 + 1):
//   Cbar_t = Cbar_{t-1} + (k k^T - Cbar_{t-1}) / t,   mu_t = mu_{t-1} + (k - mu_{t-1}) / t,
//   Sigma_t q = Cbar_t q - mu_t (mu_t . q)          (Cbar_t q alone when uncentred),
//   q_clean = q - lam Sigma_t q,
//   S_t = BackboneUpdate(S_{t-1}; k, v, gates),      o = scale S_t q_clean.
// Both backbone writes act on each row of S on its own (GLA: S[r] e^g + v_r k;
// Gated DeltaNet: alpha S[r] - alpha beta (S[r] . k) k + beta v_r k), so the
// step is two streaming passes: decode_stats_kernel updates Cbar and mu and
// forms Cbar_t q (16 rows of Cbar per workgroup), decode_out_kernel forms
// q_clean and updates 16 rows of S per workgroup, with the read.  Each cache
// element is read once and written once.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

namespace {
constexpr int kDecRows = 16;             // cache rows per workgroup
constexpr int kDecLanes = kThreads / kDecRows;  // 16 threads per row

template <typename T>
__device__ __forceinline__ float ldf(const void* p, size_t i) {
  return static_cast<float>(static_cast<const T*>(p)[i]);
}
}  // namespace

// Cbar and mu update, and Cbar_t q for rows n0 .. n0 + 15 of one head.
template <typename T, int DK>
__global__ __launch_bounds__(kThreads) void decode_stats_kernel(const DecodeArgs a) {
  constexpr int CPT = DK / kDecLanes;  // columns per thread
  const int bh = blockIdx.y;
  const int n = blockIdx.x * kDecRows + threadIdx.x / kDecLanes;
  const int c0 = (threadIdx.x % kDecLanes) * CPT;
  const float inv_t = 1.f / (float)(a.t0 + 1);
  const size_t tb = (size_t)bh * DK;
  const float kn = ldf<T>(a.k, tb + n);
  float* Crow = a.C + ((size_t)bh * DK + n) * DK + c0;
  float acc = 0.f;
#pragma unroll
  for (int c4 = 0; c4 < CPT; c4 += 4) {
    f32x4 x = *reinterpret_cast<const f32x4*>(Crow + c4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = c0 + c4 + e;
      x[e] += (kn * ldf<T>(a.k, tb + c) - x[e]) * inv_t;
      acc += x[e] * ldf<T>(a.q, tb + c);
    }
    *reinterpret_cast<f32x4*>(Crow + c4) = x;
  }
  acc = group_sum<kDecLanes>(acc);
  if (threadIdx.x % kDecLanes == 0) a.cq[tb + n] = acc;
  if (blockIdx.x == 0) {
    for (int c = threadIdx.x; c < DK; c += kThreads) {
      const float m = a.mu[tb + c];
      a.mu[tb + c] = m + (ldf<T>(a.k, tb + c) - m) * inv_t;
    }
  }
}

// q_clean, then rows v0 .. v0 + 15 of S: the backbone write and the read.
template <typename T, typename TG, int DK, bool GDN>
__global__ __launch_bounds__(kThreads) void decode_out_kernel(const DecodeArgs a) {
  constexpr int CPT = DK / kDecLanes;
  __shared__ float sQc[DK];
  __shared__ float sRed[kThreads / 64];
  const int bh = blockIdx.y;
  const int tid = threadIdx.x;
  const size_t tb = (size_t)bh * DK;

  // mu_t . q over the workgroup, then q_clean
  float mq = 0.f;
  if (a.centered)
    for (int c = tid; c < DK; c += kThreads) mq += a.mu[tb + c] * ldf<T>(a.q, tb + c);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mq += __shfl_xor(mq, off);
  if ((tid & 63) == 0) sRed[tid >> 6] = mq;
  __syncthreads();
  mq = 0.f;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) mq += sRed[w];
  const float lam = a.lam[bh];
  for (int c = tid; c < DK; c += kThreads) {
    const float sq = a.cq[tb + c] - (a.centered ? a.mu[tb + c] * mq : 0.f);
    sQc[c] = ldf<T>(a.q, tb + c) - lam * sq;
  }
  __syncthreads();

  const int r = blockIdx.x * kDecRows + tid / kDecLanes;
  const int c0 = (tid % kDecLanes) * CPT;
  const size_t vb = (size_t)bh * a.dv;
  const float vr = ldf<T>(a.v, vb + r);
  float* Srow = a.S + ((size_t)bh * a.dv + r) * DK + c0;
  f32x4 x[CPT / 4];
#pragma unroll
  for (int i = 0; i < CPT / 4; ++i) x[i] = *reinterpret_cast<const f32x4*>(Srow + 4 * i);
  float o = 0.f;
  if constexpr (GDN) {
    const float la = static_cast<const float*>(a.g)[bh];
    const float alpha = __expf(la), bt = a.beta[bh];
    float y = 0.f;  // S_{t-1}[r] . k
#pragma unroll
    for (int i = 0; i < CPT / 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) y += x[i][e] * ldf<T>(a.k, tb + c0 + 4 * i + e);
    y = group_sum<kDecLanes>(y);
    const float coef = bt * (vr - alpha * y);
#pragma unroll
    for (int i = 0; i < CPT / 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = c0 + 4 * i + e;
        x[i][e] = alpha * x[i][e] + coef * ldf<T>(a.k, tb + c);
        o += x[i][e] * sQc[c];
      }
  } else {
#pragma unroll
    for (int i = 0; i < CPT / 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = c0 + 4 * i + e;
        x[i][e] = x[i][e] * __expf(ldf<TG>(a.g, tb + c)) + vr * ldf<T>(a.k, tb + c);
        o += x[i][e] * sQc[c];
      }
  }
#pragma unroll
  for (int i = 0; i < CPT / 4; ++i) *reinterpret_cast<f32x4*>(Srow + 4 * i) = x[i];
  o = group_sum<kDecLanes>(o);
  if (tid % kDecLanes == 0) static_cast<T*>(a.o)[vb + r] = static_cast<T>(a.scale * o);
}

namespace {
template <typename T, typename TG, int DK>
hipError_t run_decode(const DecodeArgs& a, bool gdn, hipStream_t st) {
  const int bh = a.B * a.H;
  if (bh == 0) return hipSuccess;
  hipLaunchKernelGGL((decode_stats_kernel<T, DK>), dim3(DK / kDecRows, bh), dim3(kThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (gdn)
    hipLaunchKernelGGL((decode_out_kernel<T, float, DK, true>), dim3(a.dv / kDecRows, bh), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((decode_out_kernel<T, TG, DK, false>), dim3(a.dv / kDecRows, bh), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG>
hipError_t decode_dispatch(const DecodeArgs& a, bool gdn, hipStream_t st) {
  switch (a.dk) {
    case 64: return run_decode<T, TG, 64>(a, gdn, st);
    case 128: return run_decode<T, TG, 128>(a, gdn, st);
    case 256: return run_decode<T, TG, 256>(a, gdn, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

bool decode_supported(int dk, int dv) {
  return (dk == 64 || dk == 128 || dk == 256) && (dv == 64 || dv == 128 || dv == 256 || dv == 512);
}

hipError_t launch_decode(const DecodeArgs& a, bool gdn, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16)
    return gate_bf16 ? decode_dispatch<bf16_t, bf16_t>(a, gdn, st) : decode_dispatch<bf16_t, float>(a, gdn, st);
  return gate_bf16 ? decode_dispatch<float, bf16_t>(a, gdn, st) : decode_dispatch<float, float>(a, gdn, st);
}

}  // namespace ccq
