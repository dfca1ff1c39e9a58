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
  constexpr int LDQ = DK + P, LDA = C + P;
  constexpr int NTN = CT / 16;                     // column tiles of the slice
  constexpr int NPW = CT * DK / (16 * 16 * 4);     // state tiles per wave
  constexpr int RPW = (DK / 16) / 4;               // state row tiles per wave
  static_assert(NPW >= 1 && RPW >= 1 && NPW == RPW * NTN, "tile split");
  constexpr int VE = 8;
  typedef T vec_t __attribute__((ext_vector_type(VE)));

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sAh[C * LDA];  // A'[i][j]
  __shared__ __align__(16) T sAl[kSplit ? C * LDA : 8];
  __shared__ __align__(16) T sSh[CT * LDQ];  // S^K rows n0.. as B^T operand [n][c]
  __shared__ __align__(16) T sSl[kSplit ? CT * LDQ : 8];
  __shared__ __align__(16) float sM[DK];
  __shared__ float sMq[C], sCq[C], sLam[C];

  const int ntiles = DK / CT;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / ntiles;
  const int n0 = (lb % ntiles) * CT;  // first S^K column / q_clean column of this block
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* q = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  T* qc_out = static_cast<T*>(a.qclean);
  const size_t gstride = (size_t)a.H * DK;
  const float t0f = (float)a.t0;

  // carried state, transposed: tile u holds S^K[c][n], c = 16 tr + 4 g4 + r (all
  // DK rows over the waves), n = n0 + 16 tn + c16; Mt[v] holds the key sum of
  // row tile (w RPW + v) in column 0.
  f32x4 sk[NPW], Mt[RPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) {
    const int tr = w * RPW + u / NTN, tn = u % NTN;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = 16 * tr + 4 * g4 + r, n = n0 + 16 * tn + c16;
      sk[u][r] = a.C0 ? t0f * a.C0[((size_t)bh * DK + c) * DK + n] : 0.f;
    }
  }
#pragma unroll
  for (int v = 0; v < RPW; ++v)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = 16 * (w * RPW + v) + 4 * g4 + r;
      Mt[v][r] = (a.mu0 && c16 == 0) ? t0f * a.mu0[(size_t)bh * DK + c] : 0.f;
    }

  auto publish_state = [&]() {  // S^K -> sSh/sSl [n][c], key sum -> sM
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tr = w * RPW + u / NTN, tn = u % NTN;
      const int off = (16 * tn + c16) * LDQ + 16 * tr + 4 * g4;
      if constexpr (kSplit) {
        bf16_t h0, h1, h2, h3, l0, l1, l2, l3;
        split_bf16(sk[u][0], h0, l0);
        split_bf16(sk[u][1], h1, l1);
        split_bf16(sk[u][2], h2, l2);
        split_bf16(sk[u][3], h3, l3);
        *reinterpret_cast<bf16x4*>(sSh + off) = bf16x4{h0, h1, h2, h3};
        *reinterpret_cast<bf16x4*>(sSl + off) = bf16x4{l0, l1, l2, l3};
      } else {
        store4(sSh + off, sk[u][0], sk[u][1], sk[u][2], sk[u][3]);
      }
    }
    if (c16 == 0)
#pragma unroll
      for (int v = 0; v < RPW; ++v)
        *reinterpret_cast<f32x4*>(sM + 16 * (w * RPW + v) + 4 * g4) = Mt[v];
  };
  publish_state();

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
    __syncthreads();  // (A) previous chunk's readers are done with LDS
    rq.store(sQ, LDQ);
    rk.store(sK, LDQ);
    if (tid < C) sLam[tid] = rlam.get();
    if (r0 + C < a.T) prefetch(r0 + C);  // next chunk's loads overlap this chunk's math
    __syncthreads();  // (B)

    // M_r . q_i: four threads per row
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
    // transposed score tiles: sc[J][r] = k_j . q_i, j = 16 J + 4 g4 + r, i = 16 w + c16
    f32x4 sc[4];
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      sc[J] = zero4();
      if (J <= w) tile_mma<T, DK>(sc[J], sK + 16 * J * LDQ, LDQ, sQ + 16 * w * LDQ, LDQ);
    }
    __syncthreads();  // (C) sMq visible
    {
      const int i = 16 * w + c16;
      float rs = 0.f;
#pragma unroll
      for (int J = 0; J < 4; ++J)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (J <= w && 16 * J + 4 * g4 + r <= i) rs += sc[J][r];
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      const float cq = sMq[i] + rs;   // m_t . q_i (raw key sum up to t_i)
      const float it = 1.f / (t0f + (float)(r0 + i + 1));
      if (g4 == 0) sCq[i] = cq;
      if (a.mdot && n0 == 0 && g4 == 0 && i < nrow) a.mdot[((size_t)b * a.T + r0 + i) * a.H + h] = cq;
      const float mean = a.centered ? cq * it * it : 0.f;
      // A'[i][j] = (q_i . k_j)/t_i - cq_i/t_i^2 for j <= i, written as row i
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = 16 * J + 4 * g4 + r;
          x[r] = (J <= w && j <= i) ? sc[J][r] * it - mean : 0.f;
        }
        const int off = i * LDA + 16 * J + 4 * g4;
        if constexpr (kSplit) {
          bf16_t h0, h1, h2, h3, l0, l1, l2, l3;
          split_bf16(x[0], h0, l0);
          split_bf16(x[1], h1, l1);
          split_bf16(x[2], h2, l2);
          split_bf16(x[3], h3, l3);
          *reinterpret_cast<bf16x4*>(sAh + off) = bf16x4{h0, h1, h2, h3};
          *reinterpret_cast<bf16x4*>(sAl + off) = bf16x4{l0, l1, l2, l3};
        } else {
          store4(sAh + off, x[0], x[1], x[2], x[3]);
        }
      }
    }
    __syncthreads();  // (D)

    // c and q_clean for rows of stripe w, columns [n0, n0 + CT)
#pragma unroll
    for (int tn = 0; tn < NTN; ++tn) {
      f32x4 a1 = zero4(), a2 = zero4();
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32) {
        if (k0 <= 16 * w) {  // A' is zero for j > i
          const Frag<T> fb = ld_frag_tr(sK + k0 * LDQ + n0 + 16 * tn, LDQ);
          mma(a1, ld_frag(sAh + 16 * w * LDA + k0, LDA), fb);
          if constexpr (kSplit) mma(a1, ld_frag(sAl + 16 * w * LDA + k0, LDA), fb);
        }
      }
#pragma unroll
      for (int k0 = 0; k0 < DK; k0 += 32) {
        const Frag<T> fa = ld_frag(sQ + 16 * w * LDQ + k0, LDQ);
        mma(a2, fa, ld_frag(sSh + 16 * tn * LDQ + k0, LDQ));
        if constexpr (kSplit) mma(a2, fa, ld_frag(sSl + 16 * tn * LDQ + k0, LDQ));
      }
      const int col = n0 + 16 * tn + c16;
      const float mcol = a.centered ? sM[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * g4 + r;
        const float it = 1.f / (t0f + (float)(r0 + i + 1));
        const float c = a1[r] + a2[r] * it - sCq[i] * it * it * mcol;
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
    __syncthreads();  // (E) the state tile and M have been read

    // S^K_{r+1} = S^K_r + K^T K (columns n0..), M_{r+1} = M_r + sum_j k_j
    {
      const Frag<T> ones = ones_col_frag<T>();
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32) {
        Frag<T> fb[NTN];
#pragma unroll
        for (int tn = 0; tn < NTN; ++tn) fb[tn] = ld_frag_tr(sK + k0 * LDQ + n0 + 16 * tn, LDQ);
#pragma unroll
        for (int v = 0; v < RPW; ++v) {
          const Frag<T> fa = ld_frag_tr(sK + k0 * LDQ + 16 * (w * RPW + v), LDQ);
#pragma unroll
          for (int tn = 0; tn < NTN; ++tn) mma(sk[v * NTN + tn], fa, fb[tn]);
          mma(Mt[v], fa, ones);
        }
      }
    }
    publish_state();
  }
  __syncthreads();

  // final normalised statistics Cbar_T = S^K_T / t, mu_T = M_T / t
  const float tfin = t0f + (float)a.T;
  if (tfin > 0.f) {
    const float inv = 1.f / tfin;
    if (a.CT) {
#pragma unroll
      for (int u = 0; u < NPW; ++u) {
        const int tr = w * RPW + u / NTN, tn = u % NTN;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int c = 16 * tr + 4 * g4 + r, n = n0 + 16 * tn + c16;
          a.CT[((size_t)bh * DK + c) * DK + n] = sk[u][r] * inv;
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
      case 128: return run_clean<float, 128, 32>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
