// ccq_bwd.hip -- CCQ-GLA training step: gradients of L = sum_t <dO_t, o_t>.
//
// Forward (per head, scale s):  q_clean_t = (I - lam_t Sigma_t) q_t,
//   S_t = S_{t-1} diag(e^{g_t}) + v_t k_t^T,   o_t = s S_t q_clean_t.
//
// GLA part, chunk r with inclusive log-decay prefix b, entering state S_r and
// dS_{r+1} = dL/d(state leaving the chunk):
//   dS_r    = dS_{r+1} diag(e^{b_C}) + s sum_t dO_t (qc_t * e^{b_t})^T
//   dqc_t   = s e^{b_t} * [S_r^T dO_t + sum_{j<=t} (dO_t . v_j) k_j e^{-b_j}]
//   dk_j    = e^{-b_j} * [s sum_{t>=j} (dO_t . v_j) qc_t e^{b_t} + (dS_{r+1}^T v_j) e^{b_C}]
//   dv_j    = s sum_{t>=j} (qc_t . k_j e^{b_t - b_j}) dO_t + dS_{r+1} (k_j * e^{b_C - b_j})
//   dg_s    = sum_{t>=s} (qc_t * dqc_t - k_t * dk_t)     (dk: the GLA part only)
// (all exponentials taken relative to a mid-chunk reference, as in the forward).
//
// Contraction part, u_t = dqc_t:
//   dq_t    = (I - lam_t Sigma_t) u_t                     (Sigma_t is symmetric)
//   dlam_t  = -u_t . Sigma_t q_t
//   dk_j   += sum_{t>=j} rho_t [u_t (q_t . k_j) + q_t (u_t . k_j)]
//             + sum_{t>=j} (lam_t / t^2) [u_t (m_t . q_t) + q_t (m_t . u_t)],  rho_t = -lam_t / t
// where the last line is the mean term (absent in the uncentred variant).
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// ----------------------------------------------------------------------------
// Reverse scan of dS per (head, BV-row slice), storing dS_{r+1} for every chunk.
template <typename T, typename TG, int DK, int BV>
__global__ __launch_bounds__(kThreads, 1) void gla_dstate_kernel(const DstateArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDT = C + P, LDG = DK + 1;
  constexpr int NTC = DK / 16;
  constexpr int NPW = BV * DK / (16 * 16 * 4);
  static_assert(NPW >= 1 && DK <= kThreads, "tile split");

  __shared__ __align__(16) T sQeT[DK * LDT];
  __shared__ __align__(16) T sdOT[BV * LDT];
  __shared__ float sG[C * LDG];
  __shared__ float sDec[DK];

  const int nvt = a.dv / BV;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / nvt;
  const int v0 = (lb % nvt) * BV;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* qc = static_cast<const T*>(a.qc);
  const TG* gate = static_cast<const TG*>(a.g);
  const T* dO = static_cast<const T*>(a.dO);
  T* dst = static_cast<T*>(a.dstates);

  f32x4 dS[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) dS[u] = zero4();

  ChunkTile<T, DK> rq;
  ChunkTile<TG, DK> rg;
  ChunkTile<T, BV> rdo;
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rq.load(qc + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    rg.load(gate + tok_off(b, r0, h, a.T, a.H, DK), (size_t)a.H * DK, nrow);
    rdo.load(dO + tok_off(b, r0, h, a.T, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
  };
  if (N > 0) prefetch(N - 1);

  for (int ci = N - 1; ci >= 0; --ci) {
    __syncthreads();  // (A)
    rg.store_f32(sG, LDG);
    rdo.store_t(sdOT, LDT);
    {  // adjoint of the state leaving chunk ci
      T* out = dst + (((size_t)bh * N + ci) * a.dv + v0) * DK;
#pragma unroll
      for (int u = 0; u < NPW; ++u) {
        const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
#pragma unroll
        for (int r = 0; r < 4; ++r) out[(size_t)(16 * tv + 4 * g4 + r) * DK + 16 * tc + c16] = to<T>(dS[u][r]);
      }
    }
    __syncthreads();  // (B)
    if (tid < DK) {
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
    {  // (qc * e^{b})^T, e^{b} <= 1
      const int j = ChunkTile<T, DK>::row();
#pragma unroll
      for (int u = 0; u < ChunkTile<T, DK>::NV; ++u) {
        const auto x = rq.get(u);
        const int c0 = ChunkTile<T, DK>::col(u);
#pragma unroll
        for (int e = 0; e < 8; ++e) sQeT[(c0 + e) * LDT + j] = to<T>(f32(x[e]) * __expf(sG[j * LDG + c0 + e]));
      }
    }
    if (ci > 0) prefetch(ci - 1);
    __syncthreads();  // (D)
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tv = tau / NTC, tc = tau % NTC;
      f32x4 d = zero4();
      tile_mma<T, C>(d, sdOT + 16 * tv * LDT, LDT, sQeT + 16 * tc * LDT, LDT);
      const float dec = sDec[16 * tc + c16];
#pragma unroll
      for (int r = 0; r < 4; ++r) dS[u][r] = dS[u][r] * dec + a.scale * d[r];
    }
  }
}

// ----------------------------------------------------------------------------
// One workgroup per chunk: dqc, the GLA part of dk, dv, the decay gradient
// db and dlam, looping over BV-wide slices of the value dimension.
template <typename T, typename TG, int DK, int BV>
__global__ __launch_bounds__(kThreads, 1) void gla_bwd_chunk_kernel(const GlaBwdArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDT = C + P, LDG = DK + 1, LDV = BV + P;
  constexpr int NTC = DK / 16;
  constexpr int ES = (int)sizeof(T);
  static_assert(DK <= kThreads, "one thread per key channel in the scan");

  __shared__ float sG[C * LDG];  // inclusive log-decay prefix b
  __shared__ __align__(16) T sQtT[DK * LDT];
  __shared__ __align__(16) T sKtT[DK * LDT];
  __shared__ __align__(16) T sKt[C * LDQ];
  __shared__ __align__(16) T sAqkT[C * LDT];  // s (Qt Kt^T masked)^T
  __shared__ float sBm[DK], sBCm[DK];
  // phase-local buffers share one region
  constexpr int kR1 = C * LDQ * ES;
  constexpr int kOffdS = DK * LDV * ES, kOffdST = kOffdS + BV * LDQ * ES,
                kOffV = kOffdST + DK * LDV * ES, kOffdO = kOffV + C * LDV * ES,
                kOffdOT = kOffdO + C * LDV * ES, kR2 = kOffdOT + BV * LDT * ES;
  constexpr int kR3 = 2 * C * LDT * ES;
  constexpr int kR4 = 4 * DK * 4;
  constexpr int kR = kR1 > kR2 ? (kR1 > kR3 ? kR1 : kR3) : (kR2 > kR3 ? kR2 : kR3);
  __shared__ __align__(16) char sR[kR > kR4 ? kR : kR4];
  T* sQt = reinterpret_cast<T*>(sR);
  T* sSrT = reinterpret_cast<T*>(sR);
  T* sdS = reinterpret_cast<T*>(sR + kOffdS);
  T* sdST = reinterpret_cast<T*>(sR + kOffdST);
  T* sV = reinterpret_cast<T*>(sR + kOffV);
  T* sdO = reinterpret_cast<T*>(sR + kOffdO);
  T* sdOT = reinterpret_cast<T*>(sR + kOffdOT);
  T* sAdv = reinterpret_cast<T*>(sR);
  T* sAdvT = reinterpret_cast<T*>(sR + C * LDT * ES);
  float* sTot = reinterpret_cast<float*>(sR);

  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* qc = static_cast<const T*>(a.qc);
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);
  const TG* gate = static_cast<const TG*>(a.g);
  const T* dO = static_cast<const T*>(a.dO);
  const T* Sst = static_cast<const T*>(a.states) + ((size_t)bh * N + ci) * a.dv * DK;
  const T* dSst = static_cast<const T*>(a.dstates) + ((size_t)bh * N + ci) * a.dv * DK;
  const size_t gsk = (size_t)a.H * DK, gsv = (size_t)a.H * a.dv;

  // ---- phase 1: decay prefix, rescaled Qt / Kt, intra block
  {
    ChunkTile<T, DK> rq, rk;
    ChunkTile<TG, DK> rg;
    rq.load(qc + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rg.load(gate + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rg.store_f32(sG, LDG);
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
      sBCm[tid] = __expf(x[C - 1] - x[C / 2 - 1]);
    }
    __syncthreads();
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
        sQtT[(c0 + e) * LDT + j] = qo[e];
        sKtT[(c0 + e) * LDT + j] = ko[e];
      }
      *reinterpret_cast<typename ChunkTile<T, DK>::vec_t*>(sQt + j * LDQ + c0) = qo;
      *reinterpret_cast<typename ChunkTile<T, DK>::vec_t*>(sKt + j * LDQ + c0) = ko;
    }
  }
  __syncthreads();
#pragma unroll
  for (int J = 0; J < 4; ++J) {
    f32x4 acc = zero4();
    if (J <= w) tile_mma<T, DK>(acc, sQt + 16 * w * LDQ, LDQ, sKt + 16 * J * LDQ, LDQ);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * w + 4 * g4 + r, jj = 16 * J + c16;
      sAqkT[jj * LDT + i] = to<T>((J <= w && jj <= i) ? a.scale * acc[r] : 0.f);
    }
  }
  __syncthreads();  // sQt is dead from here on

  // ---- phase 2: loop over value slices
  f32x4 X1[NTC], X2[NTC], Adv[4];
#pragma unroll
  for (int ct = 0; ct < NTC; ++ct) { X1[ct] = zero4(); X2[ct] = zero4(); }
#pragma unroll
  for (int J = 0; J < 4; ++J) Adv[J] = zero4();
  T* dvout = static_cast<T*>(a.dv_out);
  for (int vv0 = 0; vv0 < a.dv; vv0 += BV) {
    // states: S_r diag(e^{b_m}) transposed, dS_{r+1} diag(e^{b_C - b_m}) and dS_{r+1}^T
    for (int idx = tid; idx < BV * DK / 8; idx += kThreads) {
      const int row = idx / (DK / 8), c0 = (idx % (DK / 8)) * 8;
      typedef T v8 __attribute__((ext_vector_type(8)));
      const v8 sv = *reinterpret_cast<const v8*>(Sst + (size_t)(vv0 + row) * DK + c0);
      const v8 dv8 = *reinterpret_cast<const v8*>(dSst + (size_t)(vv0 + row) * DK + c0);
      v8 ds_scaled;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sSrT[(c0 + e) * LDV + row] = to<T>(f32(sv[e]) * sBm[c0 + e]);
        sdST[(c0 + e) * LDV + row] = dv8[e];
        ds_scaled[e] = to<T>(f32(dv8[e]) * sBCm[c0 + e]);
      }
      *reinterpret_cast<v8*>(sdS + row * LDQ + c0) = ds_scaled;
    }
    {
      ChunkTile<T, BV> rv, rdo;
      rv.load(v + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
      rdo.load(dO + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
      rv.store(sV, LDV);
      rdo.store(sdO, LDV);
      rdo.store_t(sdOT, LDT);
    }
    __syncthreads();
#pragma unroll
    for (int ct = 0; ct < NTC; ++ct) {
      tile_mma<T, BV>(X1[ct], sdO + 16 * w * LDV, LDV, sSrT + 16 * ct * LDV, LDV);
      tile_mma<T, BV>(X2[ct], sV + 16 * w * LDV, LDV, sdST + 16 * ct * LDV, LDV);
    }
#pragma unroll
    for (int J = 0; J < 4; ++J)
      if (J <= w) tile_mma<T, BV>(Adv[J], sdO + 16 * w * LDV, LDV, sV + 16 * J * LDV, LDV);
    // dv = s (Qt Kt^T masked)^T dO + Kt (dS e^{b_C - b_m})^T  for rows of stripe w
#pragma unroll
    for (int tn = 0; tn < BV / 16; ++tn) {
      f32x4 acc = zero4();
      tile_mma<T, C>(acc, sAqkT + 16 * w * LDT, LDT, sdOT + 16 * tn * LDT, LDT);
      tile_mma<T, DK>(acc, sKt + 16 * w * LDQ, LDQ, sdS + 16 * tn * LDQ, LDQ);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int jr = 16 * w + 4 * g4 + r;
        if (jr < nrow) dvout[tok_off(b, r0 + jr, h, a.T, a.H, a.dv) + vv0 + 16 * tn + c16] = to<T>(acc[r]);
      }
    }
    __syncthreads();
  }

  // ---- phase 3: intra terms with A_dv[t][j] = dO_t . v_j (j <= t)
#pragma unroll
  for (int J = 0; J < 4; ++J)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * w + 4 * g4 + r, jj = 16 * J + c16;
      const T val = to<T>((J <= w && jj <= i) ? Adv[J][r] : 0.f);
      sAdv[i * LDT + jj] = val;
      sAdvT[jj * LDT + i] = val;
    }
  __syncthreads();
  f32x4 Y2[NTC];
#pragma unroll
  for (int ct = 0; ct < NTC; ++ct) {
    tile_mma<T, C>(X1[ct], sAdv + 16 * w * LDT, LDT, sKtT + 16 * ct * LDT, LDT);
    Y2[ct] = zero4();
    tile_mma<T, C>(Y2[ct], sAdvT + 16 * w * LDT, LDT, sQtT + 16 * ct * LDT, LDT);
  }
  __syncthreads();  // sAdv/sAdvT dead: sTot may reuse the region

  // ---- phase 4: epilogue per element (row i of stripe w, key channel c)
  T* dqc_io = static_cast<T*>(a.dqc_io);
  float tot[NTC];
  float dl[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ct = 0; ct < NTC; ++ct) {
    tot[ct] = 0.f;
    const int c = 16 * ct + c16;
    const float bm = sG[(C / 2 - 1) * LDG + c];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * w + 4 * g4 + r;
      if (i < nrow) {
        const float d = sG[i * LDG + c] - bm;
        const float dqc = a.scale * __expf(d) * X1[ct][r];
        const float dkg = __expf(-d) * (Y2[ct][r] * a.scale + X2[ct][r] * sBCm[c]);
        const size_t off = tok_off(b, r0 + i, h, a.T, a.H, DK) + c;
        const float db = f32(qc[off]) * dqc - f32(k[off]) * dkg;
        a.dqc[off] = dqc;
        dqc_io[off] = to<T>(dqc);
        a.dk_gla[off] = dkg;
        a.db[off] = db;
        tot[ct] += db;
        dl[r] -= dqc * a.corr[off];
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float s = row16_sum(dl[r]);
    const int i = 16 * w + 4 * g4 + r;
    if (c16 == 0 && i < nrow) a.dlam[((size_t)b * a.T + r0 + i) * a.H + h] = s;
  }
  // per-chunk column sums of db (for the reverse cumulative sum across chunks)
#pragma unroll
  for (int ct = 0; ct < NTC; ++ct) {
    float x = tot[ct];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if (g4 == 0) sTot[w * DK + 16 * ct + c16] = x;
  }
  __syncthreads();
  if (tid < DK)
    a.db_tot[((size_t)bh * N + ci) * DK + tid] =
        sTot[tid] + sTot[DK + tid] + sTot[2 * DK + tid] + sTot[3 * DK + tid];
}

// ----------------------------------------------------------------------------
// dg_t = sum_{s >= t} db_s: one workgroup per chunk, one thread per channel.
template <typename TG>
__global__ __launch_bounds__(kThreads) void gla_dg_kernel(const DgArgs a) {
  constexpr int C = kChunk;
  const int N = (a.T + C - 1) / C;
  const int lb = blockIdx.x;
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  TG* dg = static_cast<TG*>(a.dg);
  for (int c = threadIdx.x; c < a.dk; c += kThreads) {
    float acc = 0.f;
    for (int r = ci + 1; r < N; ++r) acc += a.db_tot[((size_t)bh * N + r) * a.dk + c];
    float x[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int jj = j < nrow ? j : nrow - 1;
      x[j] = a.db[tok_off(b, r0 + jj, h, a.T, a.H, a.dk) + c];
    }
#pragma unroll
    for (int j = C - 1; j >= 0; --j) {
      if (j < nrow) {
        acc += x[j];
        dg[tok_off(b, r0 + j, h, a.T, a.H, a.dk) + c] = static_cast<TG>(acc);
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Key gradient of the contraction: reverse scan over chunks per (head, CT
// output columns).  Carried: H = sum_{later t} rho_t (u_t q_t^T + q_t u_t^T)
// (rows n0..n0+CT as fp32 accumulators) and the mean-term vector
// D = sum_{later t} (lam_t/t^2) (u_t (m_t.q_t) + q_t (m_t.u_t)).  Within the
// chunk, with j <= t:
//   W1[t][j] = q_t . k_j - (m_t.q_t)/t     applied to rho_t u_t
//   W2[t][j] = rho_t (u_t . k_j - (m_t.u_t)/t)   applied to q_t
// so dk_j = H k_j + D + sum_{t>=j} (W1[t][j] rho_t u_t + W2[t][j] q_t).
template <typename T, int DK, int CT>
__global__ __launch_bounds__(kThreads, 1) void ccq_dk_kernel(const CcqDkArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr bool kSplit = sizeof(T) == 2;
  constexpr int LDQ = DK + P, LDT = C + P, LDA = C + P;
  constexpr int NTILE_COL = DK / 16;
  constexpr int NPW = CT * DK / (16 * 16 * 4);
  static_assert(NPW >= 1, "tile split");

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sU[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sQT[DK * LDT];
  __shared__ __align__(16) T sRUT[DK * LDT];  // (rho u)^T
  __shared__ __align__(16) T sW1h[C * LDA];   // transposed: [j][t]
  __shared__ __align__(16) T sW1l[kSplit ? C * LDA : 8];
  __shared__ __align__(16) T sW2h[C * LDA];
  __shared__ __align__(16) T sW2l[kSplit ? C * LDA : 8];
  __shared__ __align__(16) T sHh[CT * LDQ];
  __shared__ __align__(16) T sHl[kSplit ? CT * LDQ : 8];
  __shared__ float sRho[C], sMq[C], sMu[C];
  __shared__ float sD[CT];

  const int ntiles = DK / CT;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / ntiles;
  const int n0 = (lb % ntiles) * CT;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* q = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  const T* uu = static_cast<const T*>(a.u);
  T* dk_out = static_cast<T*>(a.dk_out);
  const size_t gs = (size_t)a.H * DK;

  f32x4 H[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) H[u] = zero4();
  if (tid < CT) sD[tid] = 0.f;

  ChunkTile<T, DK> rq, ru, rk;
  RowScalar rlam, rmq, rmu;
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rq.load(q + tok_off(b, r0, h, a.T, a.H, DK), gs, nrow);
    ru.load(uu + tok_off(b, r0, h, a.T, a.H, DK), gs, nrow);
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gs, nrow);
    const size_t t0i = ((size_t)b * a.T + r0) * a.H + h;
    const int row = ChunkTile<T, DK>::row();
    rlam.load(a.lam + t0i, (size_t)a.H, row, nrow);
    rmq.load(a.mdot_q + t0i, (size_t)a.H, row, nrow);
    rmu.load(a.mdot_u + t0i, (size_t)a.H, row, nrow);
  };
  if (N > 0) prefetch(N - 1);

  for (int ci = N - 1; ci >= 0; --ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    __syncthreads();  // (A)
    {
      const int j = ChunkTile<T, DK>::row();
      const float tpos = (float)(r0 + j + 1);
      const float rho = -rlam.get() / tpos;
      if (w == 0) {
        sRho[j] = rho;
        sMq[j] = a.centered ? rmq.get() / tpos : 0.f;
        sMu[j] = a.centered ? rmu.get() / tpos : 0.f;
      }
      rq.store(sQ, LDQ);
      rq.store_t(sQT, LDT);
      ru.store(sU, LDQ);
      rk.store(sK, LDQ);
#pragma unroll
      for (int u = 0; u < ChunkTile<T, DK>::NV; ++u) {
        const auto x = ru.get(u);
        const int c0 = ChunkTile<T, DK>::col(u);
#pragma unroll
        for (int e = 0; e < 8; ++e) sRUT[(c0 + e) * LDT + j] = to<T>(rho * f32(x[e]));
      }
    }
    // carried H (later chunks) as the B^T operand of the inter-chunk product
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = 16 * tr + 4 * g4 + r, c = 16 * tc + c16;
        if constexpr (kSplit) {
          bf16_t hi, lo;
          split_bf16(H[u][r], hi, lo);
          sHh[n * LDQ + c] = hi;
          sHl[n * LDQ + c] = lo;
        } else {
          sHh[n * LDQ + c] = H[u][r];
        }
      }
    }
    if (ci > 0) prefetch(ci - 1);
    __syncthreads();  // (B)

    // intra weights for pairs j <= t (row stripe w of t)
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      f32x4 s1 = zero4(), s2 = zero4();
      if (J <= w) {
        tile_mma<T, DK>(s1, sQ + 16 * w * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
        tile_mma<T, DK>(s2, sU + 16 * w * LDQ, LDQ, sK + 16 * J * LDQ, LDQ);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = 16 * w + 4 * g4 + r, jj = 16 * J + c16;
        const bool on = J <= w && jj <= t;
        const float w1 = on ? s1[r] - sMq[t] : 0.f;
        const float w2 = on ? sRho[t] * (s2[r] - sMu[t]) : 0.f;
        if constexpr (kSplit) {
          bf16_t hi, lo;
          split_bf16(w1, hi, lo);
          sW1h[jj * LDA + t] = hi;
          sW1l[jj * LDA + t] = lo;
          split_bf16(w2, hi, lo);
          sW2h[jj * LDA + t] = hi;
          sW2l[jj * LDA + t] = lo;
        } else {
          sW1h[jj * LDA + t] = w1;
          sW2h[jj * LDA + t] = w2;
        }
      }
    }
    __syncthreads();  // (C)

    // dk rows of stripe w (key index j), columns [n0, n0 + CT)
#pragma unroll
    for (int tn = 0; tn < CT / 16; ++tn) {
      f32x4 acc = zero4();
#pragma unroll
      for (int k0 = 0; k0 < DK; k0 += 32) {
        const Frag<T> fa = ld_frag(sK + 16 * w * LDQ + k0, LDQ);
        mma(acc, fa, ld_frag(sHh + 16 * tn * LDQ + k0, LDQ));
        if constexpr (kSplit) mma(acc, fa, ld_frag(sHl + 16 * tn * LDQ + k0, LDQ));
      }
      const T* rut = sRUT + (n0 + 16 * tn) * LDT;
      const T* qt = sQT + (n0 + 16 * tn) * LDT;
#pragma unroll
      for (int k0 = 0; k0 < C; k0 += 32) {
        const Frag<T> f1 = ld_frag(rut + k0, LDT), f2 = ld_frag(qt + k0, LDT);
        mma(acc, ld_frag(sW1h + 16 * w * LDA + k0, LDA), f1);
        mma(acc, ld_frag(sW2h + 16 * w * LDA + k0, LDA), f2);
        if constexpr (kSplit) {
          mma(acc, ld_frag(sW1l + 16 * w * LDA + k0, LDA), f1);
          mma(acc, ld_frag(sW2l + 16 * w * LDA + k0, LDA), f2);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int jr = 16 * w + 4 * g4 + r;
        const int col = n0 + 16 * tn + c16;
        if (jr < nrow) {
          const size_t off = tok_off(b, r0 + jr, h, a.T, a.H, DK) + col;
          dk_out[off] = to<T>(a.dk_gla[off] + acc[r] + sD[16 * tn + c16]);
        }
      }
    }
    __syncthreads();  // (D) sD and the H tile have been read

    // H += (rho u)^T q + q^T (rho u) for rows [n0, n0+CT); D += this chunk's mean terms
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = w * NPW + u, tr = tau / NTILE_COL, tc = tau % NTILE_COL;
      tile_mma<T, C>(H[u], sRUT + (n0 + 16 * tr) * LDT, LDT, sQT + 16 * tc * LDT, LDT);
      tile_mma<T, C>(H[u], sQT + (n0 + 16 * tr) * LDT, LDT, sRUT + 16 * tc * LDT, LDT);
    }
    if (tid < CT) {
      float s = 0.f;
      for (int t = 0; t < C; ++t)
        s -= sMq[t] * f32(sRUT[(n0 + tid) * LDT + t]) + sRho[t] * sMu[t] * f32(sQT[(n0 + tid) * LDT + t]);
      sD[tid] += s;
    }
  }
}

// ----------------------------------------------------------------------------
namespace {
template <typename T, typename TG, int DK, int BV>
hipError_t run_dstate(const DstateArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / BV);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_dstate_kernel<T, TG, DK, BV>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG, int DK, int BV>
hipError_t run_bwd_chunk(const GlaBwdArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_bwd_chunk_kernel<T, TG, DK, BV>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK, int CT>
hipError_t run_ccq_dk(const CcqDkArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (DK / CT);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((ccq_dk_kernel<T, DK, CT>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG>
hipError_t dstate_dispatch(const DstateArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (a.dk == 64) return run_dstate<T, TG, 64, 64>(a, st);
    if (a.dk == 128) return run_dstate<T, TG, 128, 64>(a, st);
  } else {
    if (a.dk == 64) return run_dstate<T, TG, 64, 64>(a, st);
  }
  return hipErrorInvalidValue;
}
template <typename T, typename TG>
hipError_t chunk_dispatch(const GlaBwdArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (a.dk == 64) return run_bwd_chunk<T, TG, 64, 32>(a, st);
    if (a.dk == 128) return run_bwd_chunk<T, TG, 128, 32>(a, st);
  } else {
    if (a.dk == 64) return run_bwd_chunk<T, TG, 64, 32>(a, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

bool bwd_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  if (is_bf16) return dv_ok && (dk == 64 || dk == 128);
  return dv_ok && dk == 64;
}

hipError_t launch_gla_dstate(const DstateArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? dstate_dispatch<bf16_t, bf16_t>(a, st) : dstate_dispatch<bf16_t, float>(a, st);
  return gate_bf16 ? dstate_dispatch<float, bf16_t>(a, st) : dstate_dispatch<float, float>(a, st);
}

hipError_t launch_gla_bwd_chunk(const GlaBwdArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? chunk_dispatch<bf16_t, bf16_t>(a, st) : chunk_dispatch<bf16_t, float>(a, st);
  return gate_bf16 ? chunk_dispatch<float, bf16_t>(a, st) : chunk_dispatch<float, float>(a, st);
}

hipError_t launch_gla_dg(const DgArgs& a, bool gate_bf16, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk);
  if (nblk == 0) return hipSuccess;
  if (gate_bf16)
    hipLaunchKernelGGL(gla_dg_kernel<bf16_t>, dim3(nblk), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(gla_dg_kernel<float>, dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_ccq_dk(const CcqDkArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    if (a.dk == 64) return run_ccq_dk<bf16_t, 64, 16>(a, st);
    if (a.dk == 128) return run_ccq_dk<bf16_t, 128, 32>(a, st);
  } else {
    if (a.dk == 64) return run_ccq_dk<float, 64, 16>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
