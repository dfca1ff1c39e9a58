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
  constexpr int LDQ = DK + P, LDV = BV + P, LDA = C + P, LDG = DK + 1;
  constexpr int NTV = BV / 16;                 // value tiles of the slice
  constexpr int RPW = (DK / 16) / 4;           // key row tiles of S^T per wave
  constexpr int NPW = RPW * NTV;
  static_assert(RPW >= 1 && DK <= kThreads, "tile split");

  __shared__ __align__(16) T sQt[C * LDQ];   // q e^{b - b_m}
  __shared__ __align__(16) T sKt[C * LDQ];   // k e^{b_m - b}
  __shared__ __align__(16) T sV[C * LDV];    // value slice, row-major
  __shared__ __align__(16) T sS[BV * LDQ];   // S diag(e^{b_m}) as B^T operand [v][c]
  // sG (gates, then their prefix b) is dead once Qt/Kt are built; the intra
  // block A[i][j] reuses its bytes
  constexpr int kGBytes = C * LDG * 4, kABytes = C * LDA * (int)sizeof(T);
  __shared__ __align__(16) char sGA[kGBytes > kABytes ? kGBytes : kABytes];
  float* sG = reinterpret_cast<float*>(sGA);
  T* sA = reinterpret_cast<T*>(sGA);
  __shared__ __align__(16) float sBm[DK], sDecm[DK];

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
  const size_t gstride = (size_t)a.H * DK;
  const int N = (a.T + C - 1) / C;

  // state, transposed: tile u holds S[v][c] at c = 16 (w RPW + u / NTV) + 4 g4 + r,
  // v = v0 + 16 (u % NTV) + c16
  f32x4 S[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) {
    const int tr = w * RPW + u / NTV, tv = u % NTV;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = 16 * tr + 4 * g4 + r, vv = v0 + 16 * tv + c16;
      S[u][r] = a.S0 ? a.S0[((size_t)bh * a.dv + vv) * DK + c] : 0.f;
    }
  }

  ChunkTile<T, DK> rq, rk;
  ChunkTile<TG, DK> rg;
  ChunkTile<T, BV> rv;
  auto prefetch = [&](int r0) {
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rq.load(qc + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rg.load(gate + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rv.load(v + tok_off(b, r0, h, a.T, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
  };
  if (a.T > 0) prefetch(0);

  for (int ci = 0; ci < N; ++ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    __syncthreads();  // (A) previous chunk's LDS readers are done
    rg.store_f32(sG, LDG);
    rv.store(sV, LDV);
    __syncthreads();  // (B)
    // per key channel: inclusive log-decay prefix b_j (rows >= nrow have g = 0)
    if (tid < DK) {
      float x[C];
#pragma unroll
      for (int j = 0; j < C; ++j) x[j] = sG[j * LDG + tid];
#pragma unroll
      for (int j = 1; j < C; ++j) x[j] += x[j - 1];
#pragma unroll
      for (int j = 0; j < C; ++j) sG[j * LDG + tid] = x[j];
      const float bm = x[C / 2 - 1], bC = x[C - 1];
      sBm[tid] = __expf(bm);
      sDecm[tid] = __expf(bC - bm);
    }
    __syncthreads();  // (C)
    // rescale to the mid-chunk reference: Qt = q e^{b - b_m}, Kt = k e^{b_m - b}
    {
      const int j = ChunkTile<T, DK>::row();
#pragma unroll
      for (int u = 0; u < ChunkTile<T, DK>::NV; ++u) {
        const int c0 = ChunkTile<T, DK>::col(u);
        const auto xq = rq.get(u), xk = rk.get(u);
        typename ChunkTile<T, DK>::vec_t qo, ko;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = sG[j * LDG + c0 + e] - sG[(C / 2 - 1) * LDG + c0 + e];
          qo[e] = to<T>(f32(xq[e]) * __expf(d));
          ko[e] = to<T>(f32(xk[e]) * __expf(-d));
        }
        *reinterpret_cast<typename ChunkTile<T, DK>::vec_t*>(sQt + j * LDQ + c0) = qo;
        *reinterpret_cast<typename ChunkTile<T, DK>::vec_t*>(sKt + j * LDQ + c0) = ko;
      }
    }
    if (ci + 1 < N) prefetch(r0 + C);  // registers are free: next chunk's loads overlap the math
    // entering state rescaled to the reference point, S diag(e^{b_m}), as [v][c]
    // (training: S_r itself is kept for the backward)
    T* st_out = a.states ? static_cast<T*>(a.states) + (((size_t)bh * N + ci) * a.dv + v0) * DK : nullptr;
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tr = w * RPW + u / NTV, tv = u % NTV;
      const int c = 16 * tr + 4 * g4, vv = 16 * tv + c16;
      const f32x4 bm = *reinterpret_cast<const f32x4*>(sBm + c);
      store4(sS + vv * LDQ + c, S[u][0] * bm[0], S[u][1] * bm[1], S[u][2] * bm[2], S[u][3] * bm[3]);
      if (st_out) store4(st_out + (size_t)vv * DK + c, S[u][0], S[u][1], S[u][2], S[u][3]);
    }
    __syncthreads();  // (D) sG dead, sQt/sKt/sS ready
    // intra block, transposed tiles: k_j e^{b_m-b_j} . q_i e^{b_i-b_m}, stored as A[i][j] (j <= i)
    {
      const int i = 16 * w + c16;
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        f32x4 sc = zero4();
        if (J <= w) tile_mma<T, DK>(sc, sKt + 16 * J * LDQ, LDQ, sQt + 16 * w * LDQ, LDQ);
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) x[r] = (J <= w && 16 * J + 4 * g4 + r <= i) ? sc[r] : 0.f;
        store4(sA + i * LDA + 16 * J + 4 * g4, x[0], x[1], x[2], x[3]);
      }
    }
    __syncthreads();  // (E)

    // o = Qt (S diag e^{b_m})^T + A V   for rows of stripe w, columns of the slice
#pragma unroll
    for (int tv = 0; tv < NTV; ++tv) {
      f32x4 acc = zero4();
      tile_mma<T, DK>(acc, sQt + 16 * w * LDQ, LDQ, sS + 16 * tv * LDQ, LDQ);
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32)
        if (k0 <= 16 * w) mma(acc, ld_frag(sA + 16 * w * LDA + k0, LDA), ld_frag_tr(sV + k0 * LDV + 16 * tv, LDV));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r;
        if (i < nrow) o[tok_off(b, r0 + i, h, a.T, a.H, a.dv) + v0 + 16 * tv + c16] = to<T>(a.scale * acc[r]);
      }
    }
    // S^T <- diag(e^{b_C}) S^T + diag(e^{b_C - b_m}) Kt^T V
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 32) {
      Frag<T> fb[NTV];
#pragma unroll
      for (int tv = 0; tv < NTV; ++tv) fb[tv] = ld_frag_tr(sV + k0 * LDV + 16 * tv, LDV);
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) {
        const Frag<T> fa = ld_frag_tr(sKt + k0 * LDQ + 16 * (w * RPW + rr), LDQ);
#pragma unroll
        for (int tv = 0; tv < NTV; ++tv) {
          f32x4& st = S[rr * NTV + tv];
          if (k0 == 0) {  // (S e^{b_m} + Kt^T V) e^{b_C - b_m} = S e^{b_C} + (Kt^T V) e^{b_C - b_m}
            const f32x4 bm = *reinterpret_cast<const f32x4*>(sBm + 16 * (w * RPW + rr) + 4 * g4);
#pragma unroll
            for (int r = 0; r < 4; ++r) st[r] *= bm[r];
          }
          mma(st, fa, fb[tv]);
          if (k0 + 32 >= C) {
            const f32x4 decm = *reinterpret_cast<const f32x4*>(sDecm + 16 * (w * RPW + rr) + 4 * g4);
#pragma unroll
            for (int r = 0; r < 4; ++r) st[r] *= decm[r];
          }
        }
      }
    }
  }

  if (a.ST) {
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tr = w * RPW + u / NTV, tv = u % NTV;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = 16 * tr + 4 * g4 + r, vv = v0 + 16 * tv + c16;
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
  (void)is_bf16;
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gla_fwd(const GlaArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? dispatch_gla<bf16_t, bf16_t>(a, st) : dispatch_gla<bf16_t, float>(a, st);
  return gate_bf16 ? dispatch_gla<float, bf16_t>(a, st) : dispatch_gla<float, float>(a, st);
}

}  // namespace ccq
