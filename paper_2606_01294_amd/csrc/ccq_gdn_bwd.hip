// ccq_gdn_bwd.hip -- CCQ-Gated DeltaNet training step: gradients of the
// backbone, L = sum_t <dO_t, o_t>.
//
// Forward of chunk r (see ccq_gdn.hip), entered with state S_r, Q = q_clean,
// gamma the cumulative log decay inside the chunk, G = e^gamma, Tm = (I+A)^{-1}:
//   W = V - diag(G) K S_r^T,  U = Tm diag(beta) W,
//   P_ij = e^{gamma_i - gamma_j} (q_i . k_j)  (j <= i),
//   O = s [diag(G) Q S_r^T + P U],
//   S_{r+1} = e^{gamma_C} S_r + U^T diag(e^{gamma_C - gamma}) K.
// Reverse, with dO' = s dO and D = dL/dS_{r+1} (zero after the last chunk):
//   dU = P^T dO' + diag(e^{gamma_C - gamma}) K D^T,   dR = Tm^T dU,
//   dS_r = e^{gamma_C} D + dO'^T diag(G) Q - dR^T diag(beta G) K      (sequential)
// and, chunk-parallel, with G1 = dO' S_r, G2 = dR S_r, G3 = U D,
// dPm = M o (dO' U^T) (M_ij = e^{gamma_i - gamma_j}, j <= i),
// dA = -(dR U^T) strictly below the diagonal, E = diag(beta) (M o dA):
//   dQ      = diag(G) G1 + dPm K
//   dK      = dPm^T Q + diag(e^{gamma_C - gamma}) G3 - diag(beta G) G2 + E K + E^T K
//   dV      = diag(beta) dR
//   dbeta_i = dR_i . V_i - G_i (G2_i . k_i) + sum_{j<i} (M o dA)_ij (k_i . k_j)
//   dgamma_i = G_i (G1_i . q_i) + rowsum_i(F) - colsum_i(F) - beta_i G_i (G2_i . k_i)
//              + rowsum_i(Fa) - colsum_i(Fa) - e^{gamma_C - gamma_i} (G3_i . k_i),
//     F = dPm o (Q K^T), Fa = E o (K K^T); the last row of the chunk also takes
//     sum_i e^{gamma_C - gamma_i} (G3_i . k_i) + e^{gamma_C} <D, S_r>,
//   dlogalpha_s = sum_{i >= s} dgamma_i  (inside the chunk).
// dQ is dL/dq_clean; the contraction's part of the gradients follows as for
// GLA (ccq_bwd.hip).
#include <type_traits>

#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// ----------------------------------------------------------------------------
// Per chunk: PT[j][i] = e^{gamma_i - gamma_j} (qc_i . k_j) for j <= i, else 0
// (row-major, plain order), and Tm^T with rows in acc_pos order
// (TmT[i][acc_pos(j)] = Tm[j][i]; Tm itself is stored as Tm[j][acc_pos(i)]).
template <typename T, int DK>
__global__ __launch_bounds__(kThreads) void gdn_bwd_prep_kernel(const GdnPrepArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDP = C + P;
  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sTm[C * LDP];
  __shared__ float sGam[C];

  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const size_t cidx = (size_t)bh * N + ci;
  {
    RowTile<T, DK> rq, rk;
    RowTile<T, C> rt;
    rq.load(static_cast<const T*>(a.qc) + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    rk.load(static_cast<const T*>(a.k) + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    rt.load(static_cast<const T*>(a.Tm) + cidx * C * C, (size_t)C, C);
    if (tid < C) sGam[tid] = a.gam[cidx * 5 * C + tid];
    rq.store(sQ, LDQ);
    rk.store(sK, LDQ);
    rt.store(sTm, LDP);
  }
  lds_barrier();

  // the 16 score tiles (rows i of tile I against keys of tile J) dealt to the
  // waves in turn, the ten with J <= I first; P^T stored as rows j (zero
  // tiles above the diagonal)
  T* PT = static_cast<T*>(a.PT) + cidx * C * C;
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    const int t = w + 4 * s4;
    const int I = intra_tile_row(t), J = intra_tile_col(t);
    f32x4 acc = zero4();
    if (t < 10) tile_mma<T, DK>(acc, sQ + 16 * I * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
    const int j = 16 * J + c16;
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * I + 4 * g4 + r;
      x[r] = (t < 10 && j <= i) ? acc[r] * __expf(sGam[i] - sGam[j]) : 0.f;
    }
    store4(PT + (size_t)j * C + 16 * I + 4 * g4, x[0], x[1], x[2], x[3]);
  }
  // Tm^T: 8 consecutive elements of a row per 16-byte store
  T* TmT = static_cast<T*>(a.TmT) + cidx * C * C;
  for (int idx = tid; idx < C * C / 8; idx += kThreads) {
    const int i = idx / (C / 8), p0 = (idx % (C / 8)) * 8;
    typedef T v8 __attribute__((ext_vector_type(8)));
    v8 y;
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = sTm[acc_logical(p0 + e) * LDP + acc_pos(i)];
    *reinterpret_cast<v8*>(TmT + (size_t)i * C + p0) = y;
  }
}

// ----------------------------------------------------------------------------
// Reverse scan of D = dL/dS_{r+1} over the chunks of one head.  A workgroup
// owns NPR value tiles of 16, each split over NH waves by key feature: wave
// (p, hq) keeps D^T[c][v] for its DK / NH features c of tile p in MFMA
// accumulators.  Per chunk (last to first):
//   store D;  X = diag(e^{gamma_C - gamma}) K D^T (partial over each wave's
//   features, summed over the NH waves through LDS in a fixed order);
//   dU = X + PT dO';  dR = Tm^T dU -> stored;
//   D <- e^{gamma_C} D + (G Q)^T dO' - K^T diag(beta G) dR.
// The chunk's K, G Q, PT, Tm^T and dO' slice are prefetched into registers
// one chunk ahead and staged through LDS; K and q (the bulk of it) are
// requested after the partial-sum exchange and D is stored there too, so that
// the issue of those loads and stores overlaps the chunk's products (measured
// at the 1.3B training shape: 471 -> 406 us).
template <typename T, int DK, int NPR, int NH>
__global__ __launch_bounds__(64 * NPR * NH, 1) void gdn_dstate_kernel(const GdnDstateArgs a) {
  constexpr int C = kChunk, NW = NPR * NH, NT = 64 * NW, BVS = 16 * NPR;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDP = C + P;
  constexpr int DKH = DK / NH, NCT = DKH / 16, NK = DKH / 32;
  constexpr int NTO = NT < C * BVS / 8 ? NT : C * BVS / 8;  // threads staging the dO' slice
  static_assert(NK >= 1, "key split");

  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sQ[C * LDQ];      // e^{gamma_i} qc_i
  __shared__ __align__(16) T sPT[C * LDP];
  __shared__ __align__(16) T sTT[C * LDP];     // Tm^T, rows in acc_pos order
  __shared__ __align__(16) T sdOT[BVS * LDP];  // (s dO)^T of the workgroup's values
  __shared__ __align__(16) float sCf[3][C];    // e^{gamma_C - gamma}, beta e^gamma, e^{gamma_C}
  __shared__ __align__(16) f32x4 sX[NH > 1 ? NW * 4 * 64 : 1];  // partial X of every wave

  const int nvt = a.dv / BVS;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / nvt;
  const int v0 = (lb % nvt) * BVS;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int pr = w / NH, hq = w % NH;
  const int g4 = l >> 4, c16 = l & 15;
  const int v = v0 + 16 * pr + c16;
  const int c0 = hq * DKH;  // first key feature of this wave
  const T* qc = static_cast<const T*>(a.qc);
  const T* k = static_cast<const T*>(a.k);
  const T* dO = static_cast<const T*>(a.dO);
  T* dst = static_cast<T*>(a.dstates);
  T* dRg = static_cast<T*>(a.dR);

  f32x4 D[NCT];
#pragma unroll
  for (int tc = 0; tc < NCT; ++tc) D[tc] = zero4();

  // q: with eight waves as a row tile (adjacent lanes along a row, coalesced;
  // one decay per staged vector), else one row per lane (one decay per lane,
  // fewer registers)
  constexpr bool kRowQ = NT >= 512;
  typedef typename std::conditional<kRowQ, RowTile<T, DK, NT>, ChunkTile<T, DK, NT>>::type QTile;
  constexpr int NGQ = kRowQ ? RowTile<T, DK, NT>::NV : 1;
  struct Stage {
    RowTile<T, DK, NT> rk;
    QTile rq;
    RowTile<T, C, NT> rp, rt;
    ChunkTile<T, BVS, NTO> rdo;
    float gq[NGQ];             // gamma of the staged rows of q
    RowScalar cf[3];
  };
  Stage st;
  // the chunk's two key-width tiles (big) and the rest, issued at different
  // points of the previous chunk so that their issue overlaps its products
  auto prefetch_kq = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    st.rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    st.rq.load(qc + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
  };
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    const size_t cidx = (size_t)bh * N + ci;
    st.rp.load(static_cast<const T*>(a.PT) + cidx * C * C, (size_t)C, C);
    st.rt.load(static_cast<const T*>(a.TmT) + cidx * C * C, (size_t)C, C);
    if (tid < NTO) st.rdo.load(dO + tok_off(b, r0, h, a.T, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
    if constexpr (kRowQ) {
#pragma unroll
      for (int u = 0; u < NGQ; ++u) st.gq[u] = a.gam[cidx * 5 * C + RowTile<T, DK, NT>::row(u)];
    } else {
      st.gq[0] = a.gam[cidx * 5 * C + (tid & 63)];
    }
    if (tid < C) {
      st.cf[0].load(a.gam + (cidx * 5 + 3) * C, 1, tid, C);
      st.cf[1].load(a.gam + (cidx * 5 + 1) * C, 1, tid, C);
      st.cf[2].load(a.gam + (cidx * 5 + 4) * C, 1, tid, C);
    }
  };
  if (N > 0) {
    prefetch_kq(N - 1);
    prefetch(N - 1);
  }

  for (int ci = N - 1; ci >= 0; --ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    const size_t cidx = (size_t)bh * N + ci;
    lds_barrier();  // every wave is done with the previous chunk's LDS
    st.rk.store(sK, LDQ);
    st.rp.store(sPT, LDP);
    st.rt.store(sTT, LDP);
    {
      typedef typename QTile::vec_t vq;
#pragma unroll
      for (int u = 0; u < QTile::NV; ++u) {
        int qrow;
        float eg;
        if constexpr (kRowQ) {
          qrow = RowTile<T, DK, NT>::row(u);
          eg = __expf(st.gq[u]);
        } else {
          qrow = ChunkTile<T, DK, NT>::row();
          eg = __expf(st.gq[0]);
        }
        const vq x = st.rq.get(u);
        vq y;
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = to<T>(eg * f32(x[e]));
        *reinterpret_cast<vq*>(sQ + qrow * LDQ + QTile::col(u)) = y;
      }
      const int row = ChunkTile<T, BVS, NTO>::row();
      if (tid < NTO)
#pragma unroll
        for (int u = 0; u < ChunkTile<T, BVS, NTO>::NV; ++u) {
          const auto x = st.rdo.get(u);
          const int cc = ChunkTile<T, BVS, NTO>::col(u);
#pragma unroll
          for (int e = 0; e < 8; ++e) sdOT[(cc + e) * LDP + row] = to<T>(a.scale * f32(x[e]));
        }
    }
    if (tid < C) {
#pragma unroll
      for (int q = 0; q < 3; ++q) sCf[q][tid] = st.cf[q].get();
    }
    if (ci > 0) prefetch(ci - 1);
    lds_barrier();

    // X = K D^T (D^T from the accumulators), rows scaled by e^{gamma_C - gamma_i}
    Frag<T> df[NK];
#pragma unroll
    for (int m = 0; m < NK; ++m) df[m] = acc_pair_frag<T>(D[2 * m], D[2 * m + 1]);
    f32x4 dU[4];
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      dU[I] = zero4();
#pragma unroll
      for (int m = 0; m < NK; ++m)
        mma(dU[I], ld_frag_acc(sK + 16 * I * LDQ + c0 + 32 * m, (size_t)LDQ), df[m]);
    }
    if constexpr (NH > 1) {
      // sum the NH partial products of this value tile, in a fixed order so
      // every wave of the tile holds bit-identical X
#pragma unroll
      for (int I = 0; I < 4; ++I) sX[(w * 4 + I) * 64 + l] = dU[I];
      lds_barrier();
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        f32x4 sum = sX[((pr * NH) * 4 + I) * 64 + l];
#pragma unroll
        for (int hh = 1; hh < NH; ++hh) sum += sX[((pr * NH + hh) * 4 + I) * 64 + l];
        dU[I] = sum;
      }
    }
    if (ci > 0) prefetch_kq(ci - 1);
    {  // D is the adjoint of the state leaving chunk ci (stored here, after the
       // exchange, so that its issue overlaps the products too)
      T* out = dst + (cidx * a.dv + v) * DK + c0 + 4 * g4;
#pragma unroll
      for (int tc = 0; tc < NCT; ++tc) store4(out + 16 * tc, D[tc][0], D[tc][1], D[tc][2], D[tc][3]);
    }
#pragma unroll
    for (int I = 0; I < 4; ++I) dU[I] *= *reinterpret_cast<const f32x4*>(&sCf[0][16 * I + 4 * g4]);
    // dU += PT dO'
    const Frag<T> of0 = ld_frag(sdOT + 16 * pr * LDP, LDP);
    const Frag<T> of1 = ld_frag(sdOT + 16 * pr * LDP + 32, LDP);
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      mma(dU[I], ld_frag(sPT + 16 * I * LDP, LDP), of0);
      mma(dU[I], ld_frag(sPT + 16 * I * LDP + 32, LDP), of1);
    }
    T* dRrow = dRg + tok_off(b, r0, h, a.T, a.H, a.dv) + v;
    // dR = Tm^T dU
    const Frag<T> uf0 = acc_pair_frag<T>(dU[0], dU[1]);
    const Frag<T> uf1 = acc_pair_frag<T>(dU[2], dU[3]);
    f32x4 dR[4];
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      dR[I] = zero4();
      mma(dR[I], ld_frag(sTT + 16 * I * LDP, LDP), uf0);
      mma(dR[I], ld_frag(sTT + 16 * I * LDP + 32, LDP), uf1);
    }
    if (hq == 0)
#pragma unroll
      for (int I = 0; I < 4; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = 16 * I + 4 * g4 + r;
          if (i < nrow) dRrow[i * a.H * a.dv] = to<T>(dR[I][r]);
        }
    // D <- e^{gamma_C} D + (G Q)^T dO' - K^T diag(beta G) dR
#pragma unroll
    for (int I = 0; I < 4; ++I) dR[I] *= -*reinterpret_cast<const f32x4*>(&sCf[1][16 * I + 4 * g4]);
    const Frag<T> rf0 = acc_pair_frag<T>(dR[0], dR[1]);
    const Frag<T> rf1 = acc_pair_frag<T>(dR[2], dR[3]);
    const float eC = sCf[2][0];
#pragma unroll
    for (int tc = 0; tc < NCT; ++tc) {
      D[tc] *= eC;
      mma(D[tc], ld_frag_tr(sQ + c0 + 16 * tc, LDQ), of0);
      mma(D[tc], ld_frag_tr(sQ + 32 * LDQ + c0 + 16 * tc, LDQ), of1);
      mma(D[tc], ld_frag_tr_acc(sK + c0 + 16 * tc, LDQ), rf0);
      mma(D[tc], ld_frag_tr_acc(sK + 32 * LDQ + c0 + 16 * tc, LDQ), rf1);
    }
  }
}

// ----------------------------------------------------------------------------
// One workgroup per chunk (wave w owning token rows 16 (w % 4) .. + 15): the
// C x C products Q K^T and K K^T, then a loop over BV-wide value slices
// accumulating G1 = dO' S_r, G2 = dR S_r, G3 = U D, dO' U^T and dR U^T, then
// the C x C-weighted sums and the per-element and per-row epilogue.  With
// eight waves (NW = 8) the two waves of a stripe split its key-channel tiles
// and its C x C tiles (J of the same parity as the wave's half); their
// per-row sums meet through LDS.
template <typename T, int DK, int BV, int NW>
__global__ __launch_bounds__(64 * NW, 1) void gdn_bwd_chunk_kernel(const GdnBwdArgs a) {
  constexpr int C = kChunk, NT = 64 * NW;
  constexpr int HW = NW / 4;  // waves per stripe
  constexpr int NJ = 4 / HW;  // C x C tiles J of a wave: J = HW jj + hh
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDT = C + P, LDV = BV + P;
  constexpr int NTC = DK / 16, NTW = NTC / HW;  // key-channel tiles, per wave
  constexpr int ES = (int)sizeof(T);
  static_assert(BV % 32 == 0 && DK % 32 == 0, "tiles");
  static_assert((NW == 4 || NW == 8) && NTW * HW == NTC, "wave split");

  __shared__ __align__(16) T sQ[C * LDQ];  // qc rows (kept to the end; read transposed there)
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ float sGam[C], sBeta[C], sDec[C];
  __shared__ float sColF[4][C], sColA[4][C], sRV[C];
  __shared__ float sDg[C];
  __shared__ float sRed[2][NW];
  __shared__ float sHalf[HW > 1 ? 6 : 1][C];  // the second half's per-row sums
  constexpr int kR2 = 4 * C * LDV * ES + 2 * BV * LDQ * ES;
  constexpr int kR3 = 2 * C * LDT * ES;
  constexpr int kR = kR2 > kR3 ? kR2 : kR3;
  __shared__ __align__(16) char sR[kR];

  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = lane_id();
  const int sw = w & 3, hh = w >> 2;  // stripe, half (uniform)
  const int ct0 = hh * NTW;           // this wave's first key-channel tile
  const int g4 = l >> 4, c16 = l & 15;
  const size_t cidx = (size_t)bh * N + ci;
  const size_t gsk = (size_t)a.H * DK, gsv = (size_t)a.H * a.dv;
  const float eC = a.gam[(cidx * 5 + 4) * C];

  // ---- phase 1: Q K^T and K K^T (rows of stripe sw, this wave's tiles J <= sw)
  f32x4 QK[NJ], KK[NJ];
  {
    ChunkTile<T, DK, NT> rq, rk;
    rq.load(static_cast<const T*>(a.qc) + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rk.load(static_cast<const T*>(a.k) + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    if (tid < C) {
      sGam[tid] = a.gam[cidx * 5 * C + tid];
      sBeta[tid] = a.gam[(cidx * 5 + 2) * C + tid];
      sDec[tid] = a.gam[(cidx * 5 + 3) * C + tid];
    }
    rq.store(sQ, LDQ);
    rk.store(sK, LDQ);
    lds_barrier();
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      const int J = HW * jj + hh;
      QK[jj] = zero4();
      KK[jj] = zero4();
      if (J <= sw) {
        tile_mma<T, DK>(QK[jj], sQ + 16 * sw * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
        tile_mma<T, DK>(KK[jj], sK + 16 * sw * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
      }
    }
  }

  // ---- phase 2: value slices
  f32x4 G1[NTW], G2[NTW], G3[NTW], dP[NJ], dA[NJ];
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) { G1[ct] = zero4(); G2[ct] = zero4(); G3[ct] = zero4(); }
#pragma unroll
  for (int jj = 0; jj < NJ; ++jj) { dP[jj] = zero4(); dA[jj] = zero4(); }
  float rv = 0.f, dss = 0.f;
  // the slices of dO, dR and V: 8-element pieces, four per row
  typedef RowTile<T, BV, NT> VTile;
  static_assert(VTile::NV == 1, "one piece per thread");
  const int vrow = VTile::row(0), vcol = VTile::col(0);
  {
    T* sdO = reinterpret_cast<T*>(sR);
    T* sdR = sdO + C * LDV;
    T* sU = sdR + C * LDV;
    T* sV = sU + C * LDV;
    T* sS = sV + C * LDV;     // S_r slice, rows v (read transposed by the products)
    T* sD = sS + BV * LDQ;    // D slice, rows v
    const T* Sg = static_cast<const T*>(a.states) + cidx * a.dv * DK;
    const T* Ug = static_cast<const T*>(a.U) + cidx * a.dv * C;
    const T* Dg = static_cast<const T*>(a.dstates) + cidx * a.dv * DK;
    T* dvrow = static_cast<T*>(a.dv_out) + tok_off(b, r0, h, a.T, a.H, a.dv);
    typedef T v8 __attribute__((ext_vector_type(8)));
    // every value slice's global operands are requested one slice ahead
    constexpr int NPS = BV * DK / 8 / NT;              // pieces of S_r and of D per thread
    constexpr int TPU = BV * C / 8;                    // pieces of U^T
    constexpr int NPU = (TPU + NT - 1) / NT;           // per thread
    static_assert(NPS >= 1 && BV * DK / 8 % NT == 0, "piece split");
    struct Slice {
      v8 s[NPS], d[NPS], u[NPU];
      VTile rdo, rdr, rvv;
    };
    auto load_slice = [&](Slice& sl, int vv0) {
#pragma unroll
      for (int p = 0; p < NPS; ++p) {
        const int q = tid + p * NT;
        const int vt = q / (2 * DK), rem = q % (2 * DK);
        const int m = rem / 64, vr = (rem % 64) / 4, pp = rem % 4;
        sl.s[p] = *reinterpret_cast<const v8*>(Sg + (size_t)(vv0 / 16 + vt) * 16 * DK + (size_t)(m * 16 + vr) * 32 + 8 * pp);
        const int vd = q / (DK / 8), cd = (q % (DK / 8)) * 8;
        sl.d[p] = *reinterpret_cast<const v8*>(Dg + (size_t)(vv0 + vd) * DK + cd);
      }
#pragma unroll
      for (int p = 0; p < NPU; ++p) {
        const int q = tid + p * NT;
        if (TPU % NT == 0 || q < TPU) {
          const int vt = q / 128, rem = q % 128;
          const int m = rem / 64, vr = (rem % 64) / 4, pp = rem % 4;
          sl.u[p] = *reinterpret_cast<const v8*>(Ug + (size_t)(vv0 / 16 + vt) * 16 * C + (size_t)(m * 16 + vr) * 32 + 8 * pp);
        }
      }
      sl.rdo.load(static_cast<const T*>(a.dO) + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
      sl.rdr.load(static_cast<const T*>(a.dR) + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
      sl.rvv.load(static_cast<const T*>(a.v) + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
    };
    Slice cur;
    load_slice(cur, 0);
    for (int vv0 = 0; vv0 < a.dv; vv0 += BV) {
      if (VTile::mine(0)) {
        const float bt = sBeta[vrow];
        const v8 xo = cur.rdo.get(0), xr = cur.rdr.get(0), xv = cur.rvv.get(0);
        v8 yo, yd;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          yo[e] = to<T>(a.scale * f32(xo[e]));
          yd[e] = to<T>(bt * f32(xr[e]));
          rv += f32(xr[e]) * f32(xv[e]);
        }
        *reinterpret_cast<v8*>(sdO + vrow * LDV + vcol) = yo;
        *reinterpret_cast<v8*>(sdR + vrow * LDV + vcol) = xr;
        *reinterpret_cast<v8*>(sV + vrow * LDV + vcol) = xv;
        if (vrow < nrow) *reinterpret_cast<v8*>(dvrow + vrow * (int)gsv + vv0 + vcol) = yd;
      }
      // S_r and U^T slices (fragment-native: per value tile and 32-wide k
      // block, 16 rows of 32; S_r rows in natural order, U^T rows in acc_pos
      // order) and D (plain rows)
#pragma unroll
      for (int p = 0; p < NPS; ++p) {
        const int q = tid + p * NT;
        const int vt = q / (2 * DK), rem = q % (2 * DK);
        const int m = rem / 64, vr = (rem % 64) / 4, pp = rem % 4;
        const int vl = 16 * vt + vr;
        *reinterpret_cast<v8*>(sS + vl * LDQ + 32 * m + 8 * pp) = cur.s[p];
        const int vd = q / (DK / 8), cd = (q % (DK / 8)) * 8;
        *reinterpret_cast<v8*>(sD + vd * LDQ + cd) = cur.d[p];
      }
#pragma unroll
      for (int p = 0; p < NPU; ++p) {
        const int q = tid + p * NT;
        if (TPU % NT == 0 || q < TPU) {
          const int vt = q / 128, rem = q % 128;
          const int m = rem / 64, vr = (rem % 64) / 4, pp = rem % 4;
          const int vl = 16 * vt + vr;
#pragma unroll
          for (int e = 0; e < 8; ++e) sU[(32 * m + acc_logical(8 * pp + e)) * LDV + vl] = cur.u[p][e];
        }
      }
      if (vv0 + BV < a.dv) load_slice(cur, vv0 + BV);
      lds_barrier();
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj) {
        const int J = HW * jj + hh;
        if (J <= sw) {
          tile_mma<T, BV>(dP[jj], sdO + 16 * sw * LDV, LDV, sU + 16 * J * LDV, LDV);
          tile_mma<T, BV>(dA[jj], sdR + 16 * sw * LDV, LDV, sU + 16 * J * LDV, LDV);
        }
      }
#pragma unroll
      for (int ct = 0; ct < NTW; ++ct) {
#pragma unroll
        for (int k0 = 0; k0 < BV; k0 += 32) {
          const Frag<T> fs = ld_frag_tr(sS + k0 * LDQ + 16 * (ct0 + ct), LDQ);
          mma(G1[ct], ld_frag(sdO + 16 * sw * LDV + k0, LDV), fs);
          mma(G2[ct], ld_frag(sdR + 16 * sw * LDV + k0, LDV), fs);
          mma(G3[ct], ld_frag(sU + 16 * sw * LDV + k0, LDV), ld_frag_tr(sD + k0 * LDQ + 16 * (ct0 + ct), LDQ));
        }
      }
      for (int idx = tid; idx < DK * BV / 8; idx += NT) {
        const int vl = idx / (DK / 8), c = (idx % (DK / 8)) * 8;
        const v8 xs = *reinterpret_cast<const v8*>(sS + vl * LDQ + c);
        const v8 xd = *reinterpret_cast<const v8*>(sD + vl * LDQ + c);
#pragma unroll
        for (int e = 0; e < 8; ++e) dss += f32(xs[e]) * f32(xd[e]);
      }
      lds_barrier();
    }
  }
  // dR . v per row: the row's four pieces meet in adjacent lanes
  rv += __shfl_xor(rv, 1);
  rv += __shfl_xor(rv, 2);
  if (VTile::mine(0) && (tid & 3) == 0) sRV[vrow] = rv;

  // Sigma_t q_t for this wave's rows, requested now for the epilogue
  const size_t rowoff = tok_off(b, r0, h, a.T, a.H, DK);
  float cr[NTW][4];
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      cr[ct][r] = a.corr[rowoff + (i < nrow ? i : nrow - 1) * (int)gsk + 16 * (ct0 + ct) + c16];
    }

  // ---- phase 3: C x C weights
  T* sPm = reinterpret_cast<T*>(sR);  // rows i (the products over i read it transposed)
  T* sE = sPm + C * LDT;
  float rowF[4] = {0.f, 0.f, 0.f, 0.f}, rowA[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int jj = 0; jj < NJ; ++jj) {
    const int J = HW * jj + hh;
    const int j = 16 * J + c16;
    float colF = 0.f, colA = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      const float e = (J <= sw && j <= i) ? __expf(sGam[i] - sGam[j]) : 0.f;
      const float pm = e * dP[jj][r];
      const float ea = j < i ? -e * dA[jj][r] : 0.f;  // (M o dA)_ij
      const float E = sBeta[i] * ea;
      const float F = pm * QK[jj][r];
      const float fa = ea * KK[jj][r];
      rowF[r] += F;
      rowA[r] += fa;
      colF += F;
      colA += sBeta[i] * fa;
      sPm[i * LDT + j] = to<T>(pm);
      sE[i * LDT + j] = to<T>(E);
    }
    colF += __shfl_xor(colF, 16);
    colF += __shfl_xor(colF, 32);
    colA += __shfl_xor(colA, 16);
    colA += __shfl_xor(colA, 32);
    if (g4 == 0) {
      sColF[sw][j] = colF;
      sColA[sw][j] = colA;
    }
  }
  {  // <D, S_r> over the workgroup
    float x = dss;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
    if (l == 0) sRed[0][w] = x;
  }
  lds_barrier();

  // ---- phase 4: dQ, dK and the epilogue (row i = 16 sw + 4 g4 + r, channel c)
  float dot1[4] = {0.f, 0.f, 0.f, 0.f}, dot2[4] = {0.f, 0.f, 0.f, 0.f}, dot3[4] = {0.f, 0.f, 0.f, 0.f};
  float dl[4] = {0.f, 0.f, 0.f, 0.f};
  T* dqc_io = static_cast<T*>(a.dqc_io);
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) {
    f32x4 x = zero4(), y = zero4();
    const int cc = 16 * (ct0 + ct);
    tile_mma_bt<T, C>(x, sPm + 16 * sw * LDT, LDT, sK + cc, LDQ);
    tile_mma_tr<T, C>(y, sPm + 16 * sw, LDT, sQ + cc, LDQ);
    tile_mma_bt<T, C>(y, sE + 16 * sw * LDT, LDT, sK + cc, LDQ);
    tile_mma_tr<T, C>(y, sE + 16 * sw, LDT, sK + cc, LDQ);
    const int c = cc + c16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      const float G = __expf(sGam[i]);
      const float qv = f32(sQ[i * LDQ + c]), kv = f32(sK[i * LDQ + c]);
      const float dq = G * G1[ct][r] + x[r];
      const float dk = y[r] + sDec[i] * G3[ct][r] - sBeta[i] * G * G2[ct][r];
      dot1[r] += G1[ct][r] * qv;
      dot2[r] += G2[ct][r] * kv;
      dot3[r] += G3[ct][r] * kv;
      if (i < nrow) {
        const size_t off = rowoff + i * (int)gsk + c;
        a.dqc[off] = dq;
        dqc_io[off] = to<T>(dq);
        a.dk_bb[off] = dk;
        dl[r] -= dq * cr[ct][r];
      }
    }
  }
  // per-row sums over this wave's channels (and C x C tiles); with two waves
  // per stripe the second half's sums are added through LDS
  float d1[4], d2[4], d3[4], rf[4], ra[4], dlam[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    d1[r] = row16_sum(dot1[r]);
    d2[r] = row16_sum(dot2[r]);
    d3[r] = row16_sum(dot3[r]);
    rf[r] = row16_sum(rowF[r]);
    ra[r] = row16_sum(rowA[r]);
    dlam[r] = row16_sum(dl[r]);
  }
  if constexpr (HW > 1) {
    if (hh == 1 && c16 == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * sw + 4 * g4 + r;
        sHalf[0][i] = d1[r];
        sHalf[1][i] = d2[r];
        sHalf[2][i] = d3[r];
        sHalf[3][i] = rf[r];
        sHalf[4][i] = ra[r];
        sHalf[5][i] = dlam[r];
      }
    lds_barrier();
    if (hh == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * sw + 4 * g4 + r;
        d1[r] += sHalf[0][i];
        d2[r] += sHalf[1][i];
        d3[r] += sHalf[2][i];
        rf[r] += sHalf[3][i];
        ra[r] += sHalf[4][i];
        dlam[r] += sHalf[5][i];
      }
  }
  float xt = 0.f;  // sum over this stripe's rows of e^{gamma_C - gamma_i} (G3_i . k_i)
  if (hh == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      const float G = __expf(sGam[i]), bt = sBeta[i];
      const float colF = sColF[0][i] + sColF[1][i] + sColF[2][i] + sColF[3][i];
      const float colA = sColA[0][i] + sColA[1][i] + sColA[2][i] + sColA[3][i];
      const float dg = G * d1[r] + rf[r] - colF - bt * G * d2[r] + bt * ra[r] - colA - sDec[i] * d3[r];
      if (c16 == 0) {
        sDg[i] = i < nrow ? dg : 0.f;
        xt += i < nrow ? sDec[i] * d3[r] : 0.f;
        if (i < nrow) {
          const size_t ti = ((size_t)b * a.T + r0 + i) * a.H + h;
          a.dbeta[ti] = sRV[i] - G * d2[r] + ra[r];
          a.dlam[ti] = dlam[r];
        }
      }
    }
    xt += __shfl_xor(xt, 16);
    xt += __shfl_xor(xt, 32);
    if (l == 0) sRed[1][sw] = xt;
  }
  lds_barrier();
  if (w == 0) {
    // the last row of the chunk also carries the derivative through gamma_C
    float x = sDg[l];
    if (l == nrow - 1) {
      float sd = 0.f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) sd += sRed[0][ww];
      x += (sRed[1][0] + sRed[1][1] + sRed[1][2] + sRed[1][3]) + eC * sd;
    }
    // suffix sum: dlogalpha_s = sum_{i >= s} dgamma_i
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_down(x, off);
      if (l + off < 64) x += y;
    }
    if (l < nrow) a.dlogalpha[((size_t)b * a.T + r0 + l) * a.H + h] = x;
  }
}

namespace {
template <typename T, int DK>
hipError_t run_prep(const GdnPrepArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_bwd_prep_kernel<T, DK>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK, int NPR, int NH>
hipError_t run_dstate_v(const GdnDstateArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / (16 * NPR));
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_dstate_kernel<T, DK, NPR, NH>), dim3(nblk), dim3(64 * NPR * NH), 0, st, a);
  return hipGetLastError();
}
// Value tiles per workgroup (4 or 2) and key split: with fewer value slices
// than SIMDs the features of a slice are split over two waves (measured at
// 512 slices of dk = 128: a two-way split takes 7% less time than a four-way
// one, 17% less than none), over four at dk = 256 (eight waves, two per SIMD:
// 1% less than two).
template <typename T, int DK>
hipError_t run_dstate(const GdnDstateArgs& a, hipStream_t st) {
  const long long slices = (long long)a.B * a.H * (a.dv / 16);
  if (slices >= 2048) return run_dstate_v<T, DK, 4, 1>(a, st);
  if (slices >= 1024) return run_dstate_v<T, DK, 2, 1>(a, st);
  if constexpr (DK >= 256) return run_dstate_v<T, DK, 2, 4>(a, st);
  return run_dstate_v<T, DK, 2, 2>(a, st);
}
template <typename T, int DK, int NW = 4>
hipError_t run_bwd_chunk(const GdnBwdArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk);
  if (nblk == 0) return hipSuccess;
  constexpr int BV = 32;
  hipLaunchKernelGGL((gdn_bwd_chunk_kernel<T, DK, BV, NW>), dim3(nblk), dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gdn_bwd_prep(const GdnPrepArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_prep<bf16_t, 64>(a, st);
      case 128: return run_prep<bf16_t, 128>(a, st);
      case 256: return run_prep<bf16_t, 256>(a, st);
    }
  } else if (a.dk == 64) {
    return run_prep<float, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gdn_dstate(const GdnDstateArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_dstate<bf16_t, 64>(a, st);
      case 128: return run_dstate<bf16_t, 128>(a, st);
      case 256: return run_dstate<bf16_t, 256>(a, st);
    }
  } else if (a.dk == 64) {
    return run_dstate<float, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gdn_bwd_chunk(const GdnBwdArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_bwd_chunk<bf16_t, 64>(a, st);
      case 128: return run_bwd_chunk<bf16_t, 128>(a, st);
      // eight waves at dk = 256 (the kernel takes a compute unit's LDS: two
      // waves per SIMD instead of one)
      case 256: return run_bwd_chunk<bf16_t, 256, 8>(a, st);
    }
  } else if (a.dk == 64) {
    return run_bwd_chunk<float, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
