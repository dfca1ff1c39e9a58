// ccq_clean.hip -- CCQ query contraction, chunkwise (Alg. 1 cleaning lines,
// App. B).  For every token t of chunk r (positions t = t0 + rC + i, 1-based):
//
//   c_t       = Sigma_t q_t = (1/t) K_t q_t - (1/t^2) m_t (m_t . q_t)
//   K_t       = S^K_r + sum_{rC<j<=t} k_j k_j^T   (carried state + intra block)
//   m_t       = M_r   + sum_{rC<j<=t} k_j         (carried sum + cumsum)
//   q_clean_t = q_t - lambda_t c_t                 (Eq. clean)
//
// One workgroup owns one head and a 'CT'-row slice of the symmetric S^K state
// (fp32 MFMA accumulators, carried across the sequential chunk loop) and
// produces the matching CT columns of q_clean.  Both intra-chunk terms are
// folded into one masked C x C block applied to the chunk's keys:
//
//   c_i = sum_{j<=i} A'_ij k_j + (1/t_i) S^K_r q_i - (cq_i / t_i^2) M_r,
//   A'_ij = (q_i . k_j)/t_i - cq_i/t_i^2,   cq_i = m_{t_i} . q_i = M_r.q_i + sum_{j<=i} q_i.k_j
//
// so that q_i.k_j (exact bf16 products, fp32 sums) feeds both the second-moment
// and the mean term.  fp32 operands of the bf16 products (A' and S^K) enter
// as a bf16 head plus a bf16 tail, which keeps the Cbar - mu mu^T cancellation
// (keys with a strong common mean) at ~1e-5 of |Cbar q|.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

template <typename T, int DK, int CT>
__global__ __launch_bounds__(kThreads, 1) void clean_kernel(const CleanArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr bool kSplit = sizeof(T) == 2;  // bf16: carry a tail for fp32 operands
  constexpr int LDQ = DK + P, LDT = C + P, LDA = C + P;
  constexpr int NTILE_COL = DK / 16;
  constexpr int NPW = CT * DK / (16 * 16 * 4);  // S^K tiles per wave
  static_assert(NPW >= 1, "tile split");
  constexpr int VE = 8;
  typedef T vec_t __attribute__((ext_vector_type(VE)));

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sKT[DK * LDT];
  __shared__ __align__(16) T sAh[C * LDA];
  __shared__ __align__(16) T sAl[kSplit ? C * LDA : 8];
  __shared__ __align__(16) T sSh[CT * LDQ];
  __shared__ __align__(16) T sSl[kSplit ? CT * LDQ : 8];
  __shared__ __align__(16) float sM[DK];
  __shared__ float sMq[C];
  __shared__ float sLam[C];

  const int ntiles = DK / CT;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / ntiles;
  const int n0 = (lb % ntiles) * CT;  // first S^K row / q_clean column of this block
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* q = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  T* qc_out = static_cast<T*>(a.qclean);
  const size_t gstride = (size_t)a.H * DK;
  const float t0f = (float)a.t0;

  // carried state: S^K rows [n0, n0+CT) as fp32 accumulators, M in LDS
  f32x4 sk[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) {
    const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = n0 + 16 * tr + 4 * g4 + r, c = 16 * tc + c16;
      sk[u][r] = a.C0 ? t0f * a.C0[((size_t)bh * DK + n) * DK + c] : 0.f;
    }
  }
  for (int c = tid; c < DK; c += kThreads) sM[c] = a.mu0 ? t0f * a.mu0[(size_t)bh * DK + c] : 0.f;

  auto store_state_tile = [&]() {
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = 16 * tr + 4 * g4 + r, c = 16 * tc + c16;
        if constexpr (kSplit) {
          bf16_t hi, lo;
          split_bf16(sk[u][r], hi, lo);
          sSh[n * LDQ + c] = hi;
          sSl[n * LDQ + c] = lo;
        } else {
          sSh[n * LDQ + c] = sk[u][r];
        }
      }
    }
  };
  store_state_tile();

  // chunk 0 in flight
  ChunkTile<T, DK> rq, rk;
  RowScalar rlam;
  auto prefetch = [&](int r0) {
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rq.load(q + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gstride, nrow);
    if (tid < C) rlam.load(a.lam + ((size_t)b * a.T + r0) * a.H + h, (size_t)a.H, tid, nrow);
  };
  if (a.T > 0) prefetch(0);

  for (int r0 = 0; r0 < a.T; r0 += C) {
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    __syncthreads();  // previous chunk's readers are done with LDS
    rq.store(sQ, LDQ);
    rk.store(sK, LDQ);
    rk.store_t(sKT, LDT);
    if (tid < C) sLam[tid] = rlam.get();
    if (r0 + C < a.T) prefetch(r0 + C);  // next chunk loads overlap this chunk's math
    __syncthreads();

    // M_r . q_i : four threads per row, 16-byte reads
    {
      const int row = tid >> 2, part = tid & 3;
      float s = 0.f;
#pragma unroll
      for (int c0 = part * (DK / 4); c0 < (part + 1) * (DK / 4); c0 += VE) {
        const vec_t qv = *reinterpret_cast<const vec_t*>(sQ + row * LDQ + c0);
#pragma unroll
        for (int e = 0; e < VE; ++e) s += f32(qv[e]) * sM[c0 + e];
      }
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      if (part == 0) sMq[row] = s;
    }
    // masked score block q_i . k_j for row stripe w (tiles J <= w)
    f32x4 sc[4];
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      sc[J] = zero4();
      if (J <= w) tile_mma<T, DK>(sc[J], sQ + 16 * w * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
    }
    __syncthreads();  // sMq visible
    float cq[4], inv_t[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * w + 4 * g4 + r;
      float rs = 0.f;
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        const int j = 16 * J + c16;
        if (J <= w && j <= i) rs += sc[J][r];
      }
      rs = row16_sum(rs);
      cq[r] = sMq[i] + rs;
      inv_t[r] = 1.f / (t0f + (float)(r0 + i + 1));
      if (a.mdot && n0 == 0 && c16 == 0 && i < nrow) a.mdot[((size_t)b * a.T + r0 + i) * a.H + h] = cq[r];
    }
#pragma unroll
    for (int J = 0; J < 4; ++J) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r, j = 16 * J + c16;
        float val = 0.f;
        if (J <= w && j <= i) {
          val = sc[J][r] * inv_t[r];
          if (a.centered) val -= cq[r] * inv_t[r] * inv_t[r];
        }
        if constexpr (kSplit) {
          bf16_t hi, lo;
          split_bf16(val, hi, lo);
          sAh[i * LDA + j] = hi;
          sAl[i * LDA + j] = lo;
        } else {
          sAh[i * LDA + j] = val;
        }
      }
    }
    __syncthreads();

    // c and q_clean for rows of stripe w, columns [n0, n0 + CT)
#pragma unroll
    for (int tn = 0; tn < CT / 16; ++tn) {
      f32x4 a1 = zero4(), a2 = zero4();
      const T* kt = sKT + (n0 + 16 * tn) * LDT;
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32) {
        const Frag<T> fb = ld_frag(kt + k0, LDT);
        mma(a1, ld_frag(sAh + 16 * w * LDA + k0, LDA), fb);
        if constexpr (kSplit) mma(a1, ld_frag(sAl + 16 * w * LDA + k0, LDA), fb);
      }
#pragma unroll
      for (int k0 = 0; k0 < DK; k0 += 32) {
        const Frag<T> fa = ld_frag(sQ + 16 * w * LDQ + k0, LDQ);
        mma(a2, fa, ld_frag(sSh + 16 * tn * LDQ + k0, LDQ));
        if constexpr (kSplit) mma(a2, fa, ld_frag(sSl + 16 * tn * LDQ + k0, LDQ));
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r;
        const int col = n0 + 16 * tn + c16;
        float c = a1[r] + a2[r] * inv_t[r];
        if (a.centered) c -= cq[r] * inv_t[r] * inv_t[r] * sM[col];
        if (i < nrow) {
          const size_t off = tok_off(b, r0 + i, h, a.T, a.H, DK) + col;
          const float base = a.base ? a.base[off] : f32(sQ[i * LDQ + col]);
          const float qcv = base - sLam[i] * c;
          qc_out[off] = to<T>(qcv);
          if (a.qclean_dbg) a.qclean_dbg[off] = qcv;
          if (a.corr) a.corr[off] = c;
        }
      }
    }
    __syncthreads();  // all reads of the S^K tile and of M are done

    // S^K_{r+1} = S^K_r + K^T K for rows [n0, n0+CT); M_{r+1} = M_r + sum_j k_j
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
      tile_mma<T, C>(sk[u], sKT + (n0 + 16 * tr) * LDT, LDT, sKT + 16 * tc * LDT, LDT);
    }
    store_state_tile();
    for (int c = tid; c < DK; c += kThreads) {
      float s = 0.f;
#pragma unroll
      for (int j0 = 0; j0 < C; j0 += VE) {
        const vec_t kv = *reinterpret_cast<const vec_t*>(sKT + c * LDT + j0);
#pragma unroll
        for (int e = 0; e < VE; ++e) s += f32(kv[e]);
      }
      sM[c] += s;
    }
  }
  __syncthreads();

  // final normalised statistics Cbar_T = S^K_T / t, mu_T = M_T / t
  const float tfin = t0f + (float)a.T;
  if (tfin > 0.f) {
    const float inv = 1.f / tfin;
    if (a.CT) {
#pragma unroll
      for (int u = 0; u < NPW; ++u) {
        const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = n0 + 16 * tr + 4 * g4 + r, c = 16 * tc + c16;
          a.CT[((size_t)bh * DK + n) * DK + c] = sk[u][r] * inv;
        }
      }
    }
    if (a.muT && n0 == 0)
      for (int c = tid; c < DK; c += kThreads) a.muT[(size_t)bh * DK + c] = sM[c] * inv;
  }
}

namespace {
template <typename T, int DK, int CT>
hipError_t run_clean(const CleanArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (DK / CT);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((clean_kernel<T, DK, CT>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
}  // namespace

bool clean_supported(int dk, bool is_bf16) {
  if (is_bf16) return dk == 64 || dk == 128 || dk == 256;
  return dk == 64 || dk == 128;
}

hipError_t launch_clean(const CleanArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_clean<bf16_t, 64, 16>(a, st);
      case 128: return run_clean<bf16_t, 128, 32>(a, st);
      case 256: return run_clean<bf16_t, 256, 32>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_clean<float, 64, 16>(a, st);
      case 128: return run_clean<float, 128, 16>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
