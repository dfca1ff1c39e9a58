// ccq_gla.hip -- GLA backbone chunk forward reading the cleaned queries.
//
// GLA (the cited backbone): S_t = S_{t-1} diag(e^{g_t}) + v_t k_t^T, o_t = S_t q_t.
// Within a chunk with inclusive log-decay prefix b_i = sum_{s<=i} g_s (per key
// channel) and entering state S_r:
//
//   o_i     = S_r (q_i * e^{b_i}) + sum_{j<=i} [sum_c q_i[c] k_j[c] e^{b_i[c]-b_j[c]}] v_j
//   S_{r+1} = S_r diag(e^{b_C}) + sum_j v_j (k_j * e^{b_C - b_j})^T
//
// evaluated with a mid-chunk reference m = C/2: Qt = q * e^{b - b_m},
// Kt = k * e^{b_m - b}, so that Qt Kt^T carries e^{b_i - b_j} with factors of
// at most e^{|b_m - b_i|} (a 32-token log-decay).  The inter-chunk read uses
// Qt against S diag(e^{b_m}); the state update is
// S <- S diag(e^{b_C}) + (V^T Kt) diag(e^{b_C - b_m}).
//
// One workgroup owns one head and a BV-row slice of S (fp32 MFMA accumulators
// carried over the sequential chunk loop): the rows of S evolve independently
// under the GLA write, so the slices need no communication.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

template <typename T, typename TG, int DK, int BV>
__global__ __launch_bounds__(kThreads, 1) void gla_fwd_kernel(const GlaArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDT = C + P;
  constexpr int NTC = DK / 16;
  constexpr int NPW = BV * DK / (16 * 16 * 4);
  static_assert(NPW >= 1, "tile split");
  constexpr int VE = 16 / (int)sizeof(T);
  typedef T vec_t __attribute__((ext_vector_type(VE)));

  __shared__ __align__(16) T sQt[C * LDQ];
  __shared__ __align__(16) T sKt[C * LDQ];
  __shared__ __align__(16) T sKtT[DK * LDT];
  __shared__ __align__(16) T sVT[BV * LDT];
  __shared__ __align__(16) T sA[C * LDT];
  __shared__ __align__(16) T sS[BV * LDQ];
  __shared__ float sBm[DK], sDec[DK], sDecm[DK];

  const int nvt = a.dv / BV;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / nvt;
  const int v0 = (lb % nvt) * BV;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* qc = static_cast<const T*>(a.qc);
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);
  const TG* gate = static_cast<const TG*>(a.g);
  T* o = static_cast<T*>(a.o);

  f32x4 S[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) {
    const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int vv = v0 + 16 * tv + 4 * g4 + r, c = 16 * tc + c16;
      S[u][r] = a.S0 ? a.S0[((size_t)bh * a.dv + vv) * DK + c] : 0.f;
    }
  }

  for (int r0 = 0; r0 < a.T; r0 += C) {
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    __syncthreads();
    load_chunk_rows<T, DK>(sQt, LDQ, nullptr, 0, qc + tok_off(b, r0, h, a.T, a.H, DK),
                           (size_t)a.H * DK, nrow);
    load_chunk_rows<T, DK>(sKt, LDQ, nullptr, 0, k + tok_off(b, r0, h, a.T, a.H, DK),
                           (size_t)a.H * DK, nrow);
    for (int idx = tid; idx < C * BV / VE; idx += kThreads) {
      const int row = idx / (BV / VE), c0 = (idx % (BV / VE)) * VE;
      vec_t val;
      if (row < nrow) {
        val = *reinterpret_cast<const vec_t*>(v + tok_off(b, r0 + row, h, a.T, a.H, a.dv) + v0 + c0);
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) val[e] = static_cast<T>(0.f);
      }
#pragma unroll
      for (int e = 0; e < VE; ++e) sVT[(c0 + e) * LDT + row] = val[e];
    }
    __syncthreads();

    // per key channel: inclusive log-decay prefix, reference-point rescaling
    for (int c = tid; c < DK; c += kThreads) {
      float bc[C];
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < C; ++j) {
        const float gv = j < nrow ? f32(gate[tok_off(b, r0 + j, h, a.T, a.H, DK) + c]) : 0.f;
        acc += gv;
        bc[j] = acc;
      }
      const float bm = bc[C / 2 - 1], bC = bc[C - 1];
#pragma unroll
      for (int j = 0; j < C; ++j) {
        sQt[j * LDQ + c] = to<T>(f32(sQt[j * LDQ + c]) * __expf(bc[j] - bm));
        const T kt = to<T>(f32(sKt[j * LDQ + c]) * __expf(bm - bc[j]));
        sKt[j * LDQ + c] = kt;
        sKtT[c * LDT + j] = kt;
      }
      sBm[c] = __expf(bm);
      sDec[c] = __expf(bC);
      sDecm[c] = __expf(bC - bm);
    }
    __syncthreads();

    // entering state, rescaled to the reference point: S diag(e^{b_m})
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = 16 * tv + 4 * g4 + r, c = 16 * tc + c16;
        sS[vv * LDQ + c] = to<T>(S[u][r] * sBm[c]);
      }
    }
    // intra-chunk causal block Qt Kt^T (diagonal included)
    f32x4 sc[4];
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      sc[J] = zero4();
      if (J <= w) tile_mma<T, DK>(sc[J], sQt + 16 * w * LDQ, LDQ, sKt + 16 * J * LDQ, LDQ);
    }
#pragma unroll
    for (int J = 0; J < 4; ++J)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r, j = 16 * J + c16;
        sA[i * LDT + j] = to<T>((J <= w && j <= i) ? sc[J][r] : 0.f);
      }
    __syncthreads();

    // o = Qt (S diag e^{b_m})^T + A V   for rows of stripe w, columns of the slice
#pragma unroll
    for (int tn = 0; tn < BV / 16; ++tn) {
      f32x4 acc = zero4();
      tile_mma<T, DK>(acc, sQt + 16 * w * LDQ, LDQ, sS + 16 * tn * LDQ, LDQ);
      tile_mma<T, C>(acc, sA + 16 * w * LDT, LDT, sVT + 16 * tn * LDT, LDT);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r;
        if (i < nrow) o[tok_off(b, r0 + i, h, a.T, a.H, a.dv) + v0 + 16 * tn + c16] = to<T>(a.scale * acc[r]);
      }
    }
    // S <- S diag(e^{b_C}) + (V^T Kt) diag(e^{b_C - b_m})
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
      f32x4 d = zero4();
      tile_mma<T, C>(d, sVT + 16 * tv * LDT, LDT, sKtT + 16 * tc * LDT, LDT);
      const int c = 16 * tc + c16;
      const float dec = sDec[c], decm = sDecm[c];
#pragma unroll
      for (int r = 0; r < 4; ++r) S[u][r] = S[u][r] * dec + d[r] * decm;
    }
  }

  if (a.ST) {
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = v0 + 16 * tv + 4 * g4 + r, c = 16 * tc + c16;
        a.ST[((size_t)bh * a.dv + vv) * DK + c] = S[u][r];
      }
    }
  }
}

namespace {
template <typename T, typename TG, int DK, int BV>
hipError_t run_gla(const GlaArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / BV);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_fwd_kernel<T, TG, DK, BV>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <typename T, typename TG>
hipError_t dispatch_gla(const GlaArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    switch (a.dk) {
      case 64: return run_gla<T, TG, 64, 64>(a, st);
      case 128: return run_gla<T, TG, 128, 64>(a, st);
      case 256: return run_gla<T, TG, 256, 32>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_gla<T, TG, 64, 64>(a, st);
      case 128: return run_gla<T, TG, 128, 32>(a, st);
    }
  }
  return hipErrorInvalidValue;
}
}  // namespace

bool gla_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  if (is_bf16) return dv_ok && (dk == 64 || dk == 128 || dk == 256);
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gla_fwd(const GlaArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? dispatch_gla<bf16_t, bf16_t>(a, st) : dispatch_gla<bf16_t, float>(a, st);
  return gate_bf16 ? dispatch_gla<float, bf16_t>(a, st) : dispatch_gla<float, float>(a, st);
}

}  // namespace ccq
