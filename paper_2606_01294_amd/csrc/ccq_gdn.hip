// ccq_gdn.hip -- Gated DeltaNet backbone chunk forward reading the cleaned queries.
//
// Gated DeltaNet (the cited backbone): S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T)
// + beta_t v_t k_t^T.  Writing S_t = alpha_t S_{t-1} + u_t k_t^T with
// u_t = beta_t (v_t - alpha_t S_{t-1} k_t), and gamma_i = sum_{s<=i} log alpha_s
// inside a chunk entered with state S_r, the rows u_i solve
//
//   (I + A) U = diag(beta) V - diag(beta e^gamma) K S_r^T,
//   A_ij = beta_i e^{gamma_i - gamma_j} (k_i . k_j)  (j < i),
//
// i.e. with the WY/UT factors Tm = (I + A)^{-1}, Ut = Tm diag(beta) V and
// W = Tm diag(beta e^gamma) K:  U = Ut - W S_r^T.  Then
//
//   o_i     = e^{gamma_i} S_r q_i + sum_{j<=i} e^{gamma_i - gamma_j} (k_j . q_i) u_j
//   S_{r+1} = e^{gamma_C} S_r + U^T diag(e^{gamma_C - gamma}) K.
//
// gdn_wy_kernel computes W (io dtype) and Ut (fp32) for every chunk in
// parallel; gdn_state_kernel walks the chunks of one head sequentially, owning
// a BV-row slice of S (rows of S evolve independently under this write too),
// and stores S_r and U for every chunk; gdn_out_kernel then forms the outputs
// of all chunks in parallel.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

template <typename T, int DK>
__global__ __launch_bounds__(kThreads) void gdn_wy_kernel(const WyArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P;
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) float sA[C * C];
  __shared__ float sBeta[C], sGam[C];

  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);

  {
    ChunkTile<T, DK> rk;
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    rk.store(sK, LDQ);
  }
  if (tid < C) {
    const size_t ti = ((size_t)b * a.T + r0 + tid) * a.H + h;
    float x = tid < nrow ? a.logalpha[ti] : 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(x, off);
      if (tid >= off) x += y;
    }
    sGam[tid] = x;
    sBeta[tid] = tid < nrow ? a.beta[ti] : 0.f;
  }
  __syncthreads();

  // A_ij = beta_i e^{gamma_i - gamma_j} (k_i . k_j), strictly lower
#pragma unroll
  for (int J = 0; J < 4; ++J) {
    f32x4 acc = zero4();
    if (J <= w) tile_mma<T, DK>(acc, sK + 16 * w * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * w + 4 * g4 + r, j = 16 * J + c16;
      sA[i * C + j] = (J <= w && j < i) ? sBeta[i] * __expf(sGam[i] - sGam[j]) * acc[r] : 0.f;
    }
  }
  __syncthreads();

  // forward substitution (I + A) X = R, one right-hand-side column per thread:
  // columns [0, DK) give W (R = diag(beta e^gamma) K), [DK, DK+dv) give Ut (R = diag(beta) V)
  T* Wout = static_cast<T*>(a.W) + ((size_t)bh * N + ci) * C * DK;
  float* Uout = a.Ut + ((size_t)bh * N + ci) * C * a.dv;
  for (int col = tid; col < DK + a.dv; col += kThreads) {
    float x[C];
    if (col < DK) {
#pragma unroll
      for (int i = 0; i < C; ++i) x[i] = sBeta[i] * __expf(sGam[i]) * f32(sK[i * LDQ + col]);
    } else {
      const int cv = col - DK;
#pragma unroll
      for (int i = 0; i < C; ++i)
        x[i] = i < nrow ? sBeta[i] * f32(v[tok_off(b, r0 + i, h, a.T, a.H, a.dv) + cv]) : 0.f;
    }
#pragma unroll
    for (int i = 1; i < C; ++i) {
      float s = x[i];
#pragma unroll
      for (int j = 0; j < i; ++j) s -= sA[i * C + j] * x[j];
      x[i] = s;
    }
    if (col < DK) {
#pragma unroll
      for (int i = 0; i < C; ++i) Wout[i * DK + col] = to<T>(x[i]);
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i) Uout[(size_t)i * a.dv + (col - DK)] = x[i];
    }
  }
}

// State recurrence over the chunks of one head for a BV-row slice of S:
//   S_r -> states;  U = Ut - W S_r^T -> U;  S_{r+1} = e^{gamma_C} S_r + U^T diag(e^{gamma_C - gamma}) K.
template <typename T, int DK, int BV>
__global__ __launch_bounds__(kThreads, 1) void gdn_state_kernel(const GdnArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDV = BV + P;
  constexpr int NTV = BV / 16;
  constexpr int RPW = (DK / 16) / 4;  // key row tiles of S^T per wave
  constexpr int NPW = RPW * NTV;
  static_assert(RPW >= 1, "tile split");

  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sS[BV * LDQ];   // S_r slice as [v][c]
  __shared__ __align__(16) T sUd[C * LDV];   // U[j][v] e^{gamma_C - gamma_j}
  __shared__ float sGam[C];

  const int nvt = a.dv / BV;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / nvt;
  const int v0 = (lb % nvt) * BV;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* k = static_cast<const T*>(a.k);
  const T* Wg = static_cast<const T*>(a.W);
  const size_t gstride = (size_t)a.H * DK;

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

  ChunkTile<T, DK> rk;
  RowScalar rla;
  Frag<T> rW[DK / 32];
  f32x4 rU[NTV];
  auto prefetch_k = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    if (tid < C) rla.load(a.logalpha + ((size_t)b * a.T + r0) * a.H + h, (size_t)a.H, tid, nrow);
  };
  auto prefetch_wu = [&](int ci) {
    const T* Wc = Wg + ((size_t)bh * N + ci) * C * DK + (size_t)16 * w * DK;
#pragma unroll
    for (int kk = 0; kk < DK / 32; ++kk) rW[kk] = ld_frag_global(Wc + 32 * kk, (size_t)DK);
    const float* Uc = a.Ut + (((size_t)bh * N + ci) * C + 16 * w + c16) * a.dv + v0 + 4 * g4;
#pragma unroll
    for (int tv = 0; tv < NTV; ++tv) rU[tv] = *reinterpret_cast<const f32x4*>(Uc + 16 * tv);
  };
  if (N > 0) {
    prefetch_k(0);
    prefetch_wu(0);
  }

  for (int ci = 0; ci < N; ++ci) {
    __syncthreads();  // (A) previous chunk's LDS readers are done
    rk.store(sK, LDQ);
    if (tid < C) {  // inclusive prefix of log alpha over the chunk (wave 0)
      float x = rla.get();
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (tid >= off) x += y;
      }
      sGam[tid] = x;
    }
    {
      T* st_out = static_cast<T*>(a.states) + (((size_t)bh * N + ci) * a.dv + v0) * DK;
#pragma unroll
      for (int u = 0; u < NPW; ++u) {
        const int tr = w * RPW + u / NTV, tv = u % NTV;
        const int off = (16 * tv + c16) * LDQ + 16 * tr + 4 * g4;
        store4(sS + off, S[u][0], S[u][1], S[u][2], S[u][3]);
        store4(st_out + (size_t)(16 * tv + c16) * DK + 16 * tr + 4 * g4, S[u][0], S[u][1], S[u][2], S[u][3]);
      }
    }
    __syncthreads();  // (B)
    if (ci + 1 < N) prefetch_k(ci + 1);
    const float gC = sGam[C - 1];
    {
      // U^T tiles for rows i of stripe w: U[i][v] = Ut[i][v] - (W S_r^T)[i][v]
      const int i = 16 * w + c16;
      const float ud = __expf(gC - sGam[i]);
      T* u_out = static_cast<T*>(a.U) + (((size_t)bh * N + ci) * C + i) * a.dv + v0 + 4 * g4;
#pragma unroll
      for (int tv = 0; tv < NTV; ++tv) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kk = 0; kk < DK / 32; ++kk) mma(acc, ld_frag(sS + 16 * tv * LDQ + 32 * kk, LDQ), rW[kk]);
        const float u0 = rU[tv][0] - acc[0], u1 = rU[tv][1] - acc[1];
        const float u2 = rU[tv][2] - acc[2], u3 = rU[tv][3] - acc[3];
        store4(u_out + 16 * tv, u0, u1, u2, u3);
        store4(sUd + i * LDV + 16 * tv + 4 * g4, u0 * ud, u1 * ud, u2 * ud, u3 * ud);
      }
      if (ci + 1 < N) prefetch_wu(ci + 1);
    }
    __syncthreads();  // (C)
    // S^T <- e^{gamma_C} S^T + K^T Ud
    const float eC = __expf(gC);
#pragma unroll
    for (int u = 0; u < NPW; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) S[u][r] *= eC;
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 32) {
      Frag<T> fb[NTV];
#pragma unroll
      for (int tv = 0; tv < NTV; ++tv) fb[tv] = ld_frag_tr(sUd + k0 * LDV + 16 * tv, LDV);
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) {
        const Frag<T> fa = ld_frag_tr(sK + k0 * LDQ + 16 * (w * RPW + rr), LDQ);
#pragma unroll
        for (int tv = 0; tv < NTV; ++tv) mma(S[rr * NTV + tv], fa, fb[tv]);
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

// Output of one chunk for a 64-wide value slice (eight waves):
//   o_i = scale * (e^{gamma_i} (S_r q_i) + sum_{j<=i} e^{gamma_i - gamma_j} (k_j . q_i) u_j)

template <typename T, int DK>
__global__ __launch_bounds__(kOutThreads, 1) void gdn_out_kernel(const GdnOutArgs a) {
  constexpr int C = kChunk, BVO = 64;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDV = BVO + P, LDA = C + P;

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sS[BVO * LDQ];  // S_r rows v0.. as [v][c]
  __shared__ __align__(16) T sU[C * LDV];
  __shared__ __align__(16) T sA[C * LDA];
  __shared__ float sGam[C];

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
  {
    ChunkTile<T, DK, kOutThreads> rq, rk, rs;
    ChunkTile<T, BVO, kOutThreads> ru;
    rq.load(static_cast<const T*>(a.qc) + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rk.load(static_cast<const T*>(a.k) + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rs.load(static_cast<const T*>(a.states) + (((size_t)bh * N + ci) * a.dv + v0) * DK, (size_t)DK, C);
    ru.load(static_cast<const T*>(a.U) + ((size_t)bh * N + ci) * C * a.dv + v0, (size_t)a.dv, C);
    rq.store(sQ, LDQ);
    rk.store(sK, LDQ);
    rs.store(sS, LDQ);
    ru.store(sU, LDV);
    if (tid < C) {
      RowScalar rla;
      rla.load(a.logalpha + ((size_t)b * a.T + r0) * a.H + h, (size_t)a.H, tid, nrow);
      float x = rla.get();
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (tid >= off) x += y;
      }
      sGam[tid] = x;
    }
  }
  __syncthreads();
  // intra block: ten lower tiles (I >= J) round-robin over the waves, six zero tiles
  {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int t = w + 8 * s;
      const int I = intra_tile_row(t), J = intra_tile_col(t);
      const int i = 16 * I + c16;
      float x[4] = {0.f, 0.f, 0.f, 0.f};
      if (t < 10) {
        f32x4 sc = zero4();
        tile_mma<T, DK>(sc, sK + 16 * J * LDQ, LDQ, sQ + 16 * I * LDQ, LDQ);
        const float gi = sGam[i];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = 16 * J + 4 * g4 + r;
          x[r] = j <= i ? sc[r] * __expf(gi - sGam[j]) : 0.f;
        }
      }
      store4(sA + i * LDA + 16 * J + 4 * g4, x[0], x[1], x[2], x[3]);
    }
  }
  __syncthreads();
  // o tiles: stripe w % 4, value tiles 2 (w / 4) and 2 (w / 4) + 1
  {
    const int st = w & 3;
    T* o = static_cast<T*>(a.o);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int tv = 2 * (w >> 2) + s;
      f32x4 a1 = zero4(), a2 = zero4();
      tile_mma<T, DK>(a1, sQ + 16 * st * LDQ, LDQ, sS + 16 * tv * LDQ, LDQ);
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32)
        if (k0 <= 16 * st) mma(a2, ld_frag(sA + 16 * st * LDA + k0, LDA), ld_frag_tr(sU + k0 * LDV + 16 * tv, LDV));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * st + 4 * g4 + r;
        if (i < nrow)
          o[tok_off(b, r0 + i, h, a.T, a.H, a.dv) + v0 + 16 * tv + c16] =
              to<T>(a.scale * (__expf(sGam[i]) * a1[r] + a2[r]));
      }
    }
  }
}

namespace {
template <typename T, int DK>
hipError_t run_wy(const WyArgs& a, hipStream_t st) {
  const int N = (a.T + kChunk - 1) / kChunk;
  const int nblk = a.B * a.H * N;
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_wy_kernel<T, DK>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK, int BV>
hipError_t run_gdn_state(const GdnArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / BV);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_state_kernel<T, DK, BV>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_gdn_out(const GdnOutArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk) * (a.dv / 64);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_out_kernel<T, DK>), dim3(nblk), dim3(kOutThreads), 0, st, a);
  return hipGetLastError();
}
}  // namespace

bool gdn_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  if (is_bf16) return dv_ok && (dk == 64 || dk == 128 || dk == 256);
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gdn_wy(const WyArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_wy<bf16_t, 64>(a, st);
      case 128: return run_wy<bf16_t, 128>(a, st);
      case 256: return run_wy<bf16_t, 256>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_wy<float, 64>(a, st);
      case 128: return run_wy<float, 128>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gdn_state(const GdnArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_gdn_state<bf16_t, 64, 64>(a, st);
      case 128: return run_gdn_state<bf16_t, 128, 64>(a, st);
      case 256: return run_gdn_state<bf16_t, 256, 32>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_gdn_state<float, 64, 64>(a, st);
      case 128: return run_gdn_state<float, 128, 32>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gdn_out(const GdnOutArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_gdn_out<bf16_t, 64>(a, st);
      case 128: return run_gdn_out<bf16_t, 128>(a, st);
      case 256: return run_gdn_out<bf16_t, 256>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_gdn_out<float, 64>(a, st);
      case 128: return run_gdn_out<float, 128>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
