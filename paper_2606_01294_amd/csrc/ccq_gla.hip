// ccq_gla.hip -- GLA backbone chunk forward reading the cleaned queries.
//
// GLA (the cited backbone): S_t = S_{t-1} diag(e^{g_t}) + v_t k_t^T, o_t = S_t q_t.
// Within a chunk with inclusive log-decay prefix b_i = sum_{s<=i} g_s (per key
// channel) and entering state S_r:
//
//   o_i     = S_r (q_i * e^{b_i}) + sum_{j<=i} [sum_c q_i[c] k_j[c] e^{b_i[c]-b_j[c]}] v_j
//   S_{r+1} = S_r diag(e^{b_C}) + sum_j v_j (k_j * e^{b_C - b_j})^T
//
// gla_state_kernel carries one 64x64 tile of S through the chunks of a head
// (rows and columns of S evolve independently under the GLA write) and
// stores S_r for every chunk; gla_out_kernel forms every chunk's outputs in
// parallel.  The output uses a mid-chunk reference m = C/2: Qt = q * e^{b - b_m},
// Kt = k * e^{b_m - b}, so Qt Kt^T carries e^{b_i - b_j} with factors of at most
// e^{|b_m - b_i|} (a 32-token log-decay), and the inter-chunk read is
// Qt (S_r diag(e^{b_m}))^T.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

template <typename T, typename TG>
__global__ __launch_bounds__(kThreads, 1) void gla_state_kernel(const GlaStateArgs a) {
  constexpr int C = kChunk, BK = 64, BV = 64;
  constexpr int P = Pad<T>::value;
  constexpr int LDK = BK + P, LDV = BV + P, LDG = BK + 1;
  constexpr int NTV = BV / 16;  // wave w owns key rows 16w..16w+15 of the tile, all value tiles

  __shared__ __align__(16) T sKd[C * LDK];  // k e^{b_C - b}
  __shared__ __align__(16) T sV[C * LDV];
  __shared__ float sG[C * LDG];
  __shared__ float sDec[BK];

  const int nkt = a.dk / BK, nvt = a.dv / BV;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / (nkt * nvt), kt = (lb / nvt) % nkt, vt = lb % nvt;
  const int c0 = kt * BK, v0 = vt * BV;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);
  const TG* gate = static_cast<const TG*>(a.g);

  // S^T tile: S[tv][r] = S[v][c], c = c0 + 16 w + 4 g4 + r, v = v0 + 16 tv + c16
  f32x4 S[NTV];
#pragma unroll
  for (int tv = 0; tv < NTV; ++tv)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = c0 + 16 * w + 4 * g4 + r, vv = v0 + 16 * tv + c16;
      S[tv][r] = a.S0 ? a.S0[((size_t)bh * a.dv + vv) * a.dk + c] : 0.f;
    }

  ChunkTile<T, BK> rk;
  ChunkTile<TG, BK> rg;
  ChunkTile<T, BV> rv;
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rk.load(k + tok_off(b, r0, h, a.T, a.H, a.dk) + c0, (size_t)a.H * a.dk, nrow);
    rg.load(gate + tok_off(b, r0, h, a.T, a.H, a.dk) + c0, (size_t)a.H * a.dk, nrow);
    rv.load(v + tok_off(b, r0, h, a.T, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
  };
  if (N > 0) prefetch(0);

  for (int ci = 0; ci < N; ++ci) {
    __syncthreads();  // (A)
    rg.store_f32(sG, LDG);
    rv.store(sV, LDV);
    {  // S_r, the state entering this chunk
      T* st = static_cast<T*>(a.states) + (((size_t)bh * N + ci) * a.dv + v0) * a.dk + c0 + 16 * w + 4 * g4;
#pragma unroll
      for (int tv = 0; tv < NTV; ++tv)
        store4(st + (size_t)(16 * tv + c16) * a.dk, S[tv][0], S[tv][1], S[tv][2], S[tv][3]);
    }
    __syncthreads();  // (B)
    if (tid < BK) {  // inclusive log-decay prefix of key channel c0 + tid
      float x[C];
#pragma unroll
      for (int j = 0; j < C; ++j) x[j] = sG[j * LDG + tid];
#pragma unroll
      for (int j = 1; j < C; ++j) x[j] += x[j - 1];
#pragma unroll
      for (int j = 0; j < C; ++j) sG[j * LDG + tid] = x[j];
      sDec[tid] = __expf(x[C - 1]);
    }
    __syncthreads();  // (C)
    {
      const int j = ChunkTile<T, BK>::row();
#pragma unroll
      for (int u = 0; u < ChunkTile<T, BK>::NV; ++u) {
        const int cc = ChunkTile<T, BK>::col(u);
        const auto xk = rk.get(u);
        typename ChunkTile<T, BK>::vec_t ko;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          ko[e] = to<T>(f32(xk[e]) * __expf(sG[(C - 1) * LDG + cc + e] - sG[j * LDG + cc + e]));
        *reinterpret_cast<typename ChunkTile<T, BK>::vec_t*>(sKd + j * LDK + cc) = ko;
      }
    }
    if (ci + 1 < N) prefetch(ci + 1);
    __syncthreads();  // (D)
    // S^T <- diag(e^{b_C}) S^T + Kd^T V
    {
      const f32x4 dec = *reinterpret_cast<const f32x4*>(sDec + 16 * w + 4 * g4);
#pragma unroll
      for (int tv = 0; tv < NTV; ++tv)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[tv][r] *= dec[r];
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32) {
        const Frag<T> fa = ld_frag_tr(sKd + k0 * LDK + 16 * w, LDK);
#pragma unroll
        for (int tv = 0; tv < NTV; ++tv) mma(S[tv], fa, ld_frag_tr(sV + k0 * LDV + 16 * tv, LDV));
      }
    }
  }

  if (a.ST) {
#pragma unroll
    for (int tv = 0; tv < NTV; ++tv)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = c0 + 16 * w + 4 * g4 + r, vv = v0 + 16 * tv + c16;
        a.ST[((size_t)bh * a.dv + vv) * a.dk + c] = S[tv][r];
      }
  }
}

// Outputs of one chunk for a 64-wide value slice (eight waves):
//   o = scale * (Qt (S_r diag e^{b_m})^T + (Qt Kt^T masked) V)
template <typename T, typename TG, int DK>
__global__ __launch_bounds__(kOutThreads, 1) void gla_out_kernel(const GlaOutArgs a) {
  constexpr int C = kChunk, BVO = 64;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDV = BVO + P, LDA = C + P, LDG = DK + 1;
  static_assert(DK <= kOutThreads, "one thread per key channel in the scan");

  __shared__ __align__(16) T sQt[C * LDQ];
  __shared__ __align__(16) T sKt[C * LDQ];
  __shared__ __align__(16) T sS[BVO * LDQ];
  __shared__ __align__(16) T sV[C * LDV];
  constexpr int kGBytes = C * LDG * 4, kABytes = C * LDA * (int)sizeof(T);
  __shared__ __align__(16) char sGA[kGBytes > kABytes ? kGBytes : kABytes];
  float* sG = reinterpret_cast<float*>(sGA);  // gates, then their prefix b
  T* sA = reinterpret_cast<T*>(sGA);          // intra block, once sG is dead
  __shared__ __align__(16) float sBm[DK];

  const int nvt = a.dv / BVO;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int vt = lb % nvt, ci = (lb / nvt) % N, bh = lb / (nvt * N);
  const int v0 = vt * BVO;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int tid = threadIdx.x, w = tid >> 6, l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const size_t gstride = (size_t)a.H * DK;

  ChunkTile<T, DK, kOutThreads> rq, rk, rs;
  ChunkTile<TG, DK, kOutThreads> rg;
  {
    ChunkTile<T, BVO, kOutThreads> rv;
    rq.load(static_cast<const T*>(a.qc) + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rk.load(static_cast<const T*>(a.k) + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rg.load(static_cast<const TG*>(a.g) + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rs.load(static_cast<const T*>(a.states) + (((size_t)bh * N + ci) * a.dv + v0) * DK, (size_t)DK, C);
    rv.load(static_cast<const T*>(a.v) + tok_off(b, r0, h, a.T, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
    rg.store_f32(sG, LDG);
    rv.store(sV, LDV);
  }
  __syncthreads();
  if (tid < DK) {
    float x[C];
#pragma unroll
    for (int j = 0; j < C; ++j) x[j] = sG[j * LDG + tid];
#pragma unroll
    for (int j = 1; j < C; ++j) x[j] += x[j - 1];
#pragma unroll
    for (int j = 0; j < C; ++j) sG[j * LDG + tid] = x[j];
    sBm[tid] = __expf(x[C / 2 - 1]);
  }
  __syncthreads();
  {
    const int j = ChunkTile<T, DK, kOutThreads>::row();
#pragma unroll
    for (int u = 0; u < ChunkTile<T, DK, kOutThreads>::NV; ++u) {
      const int cc = ChunkTile<T, DK, kOutThreads>::col(u);
      const auto xq = rq.get(u), xk = rk.get(u), xs = rs.get(u);
      typename ChunkTile<T, DK, kOutThreads>::vec_t qo, ko, so;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = sG[j * LDG + cc + e] - sG[(C / 2 - 1) * LDG + cc + e];
        qo[e] = to<T>(f32(xq[e]) * __expf(d));
        ko[e] = to<T>(f32(xk[e]) * __expf(-d));
        so[e] = to<T>(f32(xs[e]) * sBm[cc + e]);  // row j of the tile is value v0 + j
      }
      *reinterpret_cast<typename ChunkTile<T, DK, kOutThreads>::vec_t*>(sQt + j * LDQ + cc) = qo;
      *reinterpret_cast<typename ChunkTile<T, DK, kOutThreads>::vec_t*>(sKt + j * LDQ + cc) = ko;
      *reinterpret_cast<typename ChunkTile<T, DK, kOutThreads>::vec_t*>(sS + j * LDQ + cc) = so;
    }
  }
  __syncthreads();  // sG is dead from here on
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int t = w + 8 * s;
    const int I = intra_tile_row(t), J = intra_tile_col(t);
    const int i = 16 * I + c16;
    float x[4] = {0.f, 0.f, 0.f, 0.f};
    if (t < 10) {
      f32x4 sc = zero4();
      tile_mma<T, DK>(sc, sKt + 16 * J * LDQ, LDQ, sQt + 16 * I * LDQ, LDQ);
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] = (16 * J + 4 * g4 + r <= i) ? sc[r] : 0.f;
    }
    store4(sA + i * LDA + 16 * J + 4 * g4, x[0], x[1], x[2], x[3]);
  }
  __syncthreads();
  {
    const int st = w & 3;
    T* o = static_cast<T*>(a.o);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int tv = 2 * (w >> 2) + s;
      f32x4 acc = zero4();
      tile_mma<T, DK>(acc, sQt + 16 * st * LDQ, LDQ, sS + 16 * tv * LDQ, LDQ);
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32)
        if (k0 <= 16 * st) mma(acc, ld_frag(sA + 16 * st * LDA + k0, LDA), ld_frag_tr(sV + k0 * LDV + 16 * tv, LDV));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * st + 4 * g4 + r;
        if (i < nrow) o[tok_off(b, r0 + i, h, a.T, a.H, a.dv) + v0 + 16 * tv + c16] = to<T>(a.scale * acc[r]);
      }
    }
  }
}

namespace {
template <typename T, typename TG>
hipError_t run_gla_state(const GlaStateArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dk / 64) * (a.dv / 64);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_state_kernel<T, TG>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG>
hipError_t run_gla_out(const GlaOutArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk) * (a.dv / 64);
  if (nblk == 0) return hipSuccess;
  if (a.dk == 64)
    hipLaunchKernelGGL((gla_out_kernel<T, TG, 64>), dim3(nblk), dim3(kOutThreads), 0, st, a);
  else if (a.dk == 128)
    hipLaunchKernelGGL((gla_out_kernel<T, TG, 128>), dim3(nblk), dim3(kOutThreads), 0, st, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}
}  // namespace

bool gla_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  (void)is_bf16;
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gla_state(const GlaStateArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? run_gla_state<bf16_t, bf16_t>(a, st) : run_gla_state<bf16_t, float>(a, st);
  return gate_bf16 ? run_gla_state<float, bf16_t>(a, st) : run_gla_state<float, float>(a, st);
}

hipError_t launch_gla_out(const GlaOutArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? run_gla_out<bf16_t, bf16_t>(a, st) : run_gla_out<bf16_t, float>(a, st);
  return gate_bf16 ? run_gla_out<float, bf16_t>(a, st) : run_gla_out<float, float>(a, st);
}

}  // namespace ccq
