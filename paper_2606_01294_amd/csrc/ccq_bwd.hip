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
// The sum over the later chunks is not accumulated token by token: the decay
// gradient at the first token of chunk r + 1 equals, per key channel c,
//   dg_{(r+1)C}[c] = sum_v S_{r+1}[c, v] dS_{r+1}[c, v]
//                  = e^{b_C[c]} sum_v S_r[c, v] dS_{r+1}[c, v] + sum_j k_j[c] dk_j^inter[c],
// (the gradient of a gate is the state it multiplies times that state's
// adjoint), with dk_j^inter = e^{b_C - b_j} * (dS_{r+1}^T v_j) the inter-chunk
// part of dk_j; every term is formed from the chunk's own operands, so the
// rounding errors of the bf16 states and products enter once per chunk
// instead of adding up over the whole sequence.
//
// Contraction part, u_t = dqc_t:
//   dq_t    = (I - lam_t Sigma_t) u_t                     (Sigma_t is symmetric)
//   dlam_t  = -u_t . Sigma_t q_t
//   dk_j   += sum_{t>=j} rho_t [u_t (q_t . k_j) + q_t (u_t . k_j)]
//             + sum_{t>=j} (lam_t / t^2) [u_t (m_t . q_t) + q_t (m_t . u_t)],  rho_t = -lam_t / t
// where the last line is the mean term (absent in the uncentred variant).
//
// The reverse scan of dS (first line) is the GLA state kernel run backwards
// (ccq_gla.hip); this file holds the chunk-parallel gradients, the decay
// gradient (each chunk's rows summed in reverse from the value at the next
// chunk's first token) and the contraction's key gradient.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// ----------------------------------------------------------------------------
// One workgroup per chunk: dqc, the GLA part of dk, dv, the decay gradient
// db, dlam and the decay gradient at the next chunk's first token, looping
// over BV-wide slices of the value dimension.  Wave w owns the 16-row stripe
// w % 4 of the chunk; with eight waves (NW = 8) the two waves of a stripe
// split its key-channel tiles (and the stripe's dO V^T tiles, the dv tiles
// and the intra block's tiles), so that every SIMD holds two waves.
template <typename T, typename TG, int DK, int BV, int NW>
__global__ __launch_bounds__(64 * NW, 1) void gla_bwd_chunk_kernel(const GlaBwdArgs a) {
  constexpr int C = kChunk, NT = 64 * NW;
  constexpr int HW = NW / 4;  // waves per stripe
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDT = C + P, LDG = DK + 1, LDV = BV + P;
  constexpr int NTC = DK / 16, NTW = NTC / HW;  // key-channel tiles, per wave
  constexpr int ES = (int)sizeof(T);
  static_assert((NW == 4 || NW == 8) && NTW * HW == NTC && (BV / 16) % HW == 0, "wave split");
  static_assert(DK <= NT, "one thread per key channel in the scan");

  __shared__ float sG[C * LDG];  // inclusive log-decay prefix b
  // the rescaled Qt and Kt stay as row-major tiles to the end: the products
  // over the chunk index take them with transposing reads
  __shared__ __align__(16) T sQt[C * LDQ];
  __shared__ __align__(16) T sKt[C * LDQ];
  __shared__ __align__(16) T sAqkT[C * LDT];  // s (Qt Kt^T masked)^T
  __shared__ float sBm[DK], sBCm[DK];
  __shared__ float sDl[HW > 1 ? C : 1];  // the second half's share of dlam
  // phase-local buffers share one region
  constexpr int kOffdS = BV * LDQ * ES, kOffV = kOffdS + BV * LDQ * ES,
                kOffdO = kOffV + C * LDV * ES, kR2 = kOffdO + C * LDV * ES;
  constexpr int kR3 = C * LDT * ES;
  constexpr int kR4 = (4 + NW) * DK * 4;
  constexpr int kR = kR2 > kR3 ? kR2 : kR3;
  __shared__ __align__(16) char sR[kR > kR4 ? kR : kR4];
  T* sS = reinterpret_cast<T*>(sR);  // S_r diag(e^{b_m}) slice, rows v
  T* sdS = reinterpret_cast<T*>(sR + kOffdS);  // dS_{r+1} diag(e^{b_C - b_m}) slice, rows v
  T* sV = reinterpret_cast<T*>(sR + kOffV);
  T* sdO = reinterpret_cast<T*>(sR + kOffdO);
  T* sAdv = reinterpret_cast<T*>(sR);  // rows t (the products over t read it transposed)
  float* sTot = reinterpret_cast<float*>(sR);

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
  const T* qc = static_cast<const T*>(a.qc);
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);
  const TG* gate = static_cast<const TG*>(a.g);
  const T* dO = static_cast<const T*>(a.dO);
  const T* Sst = static_cast<const T*>(a.states) + ((size_t)bh * N + ci) * a.dv * DK;
  const T* dSst = static_cast<const T*>(a.dstates) + ((size_t)bh * N + ci) * a.dv * DK;
  const size_t gsk = (size_t)a.H * DK, gsv = (size_t)a.H * a.dv;

  // ---- phase 1: decay prefix, rescaled Qt / Kt, intra block (the chunk's
  // rows loaded as row tiles: adjacent lanes along a row)
  {
    typedef RowTile<T, DK, NT> TileQ;
    TileQ rq, rk;
    RowTile<TG, DK, NT> rg;
    rq.load(qc + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rk.load(k + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rg.load(gate + tok_off(b, r0, h, a.T, a.H, DK), gsk, nrow);
    rg.store_f32(sG, LDG);
    lds_barrier();
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
    lds_barrier();
#pragma unroll
    for (int u = 0; u < TileQ::NV; ++u) {
      if (!TileQ::mine(u)) continue;
      const int j = TileQ::row(u), c0 = TileQ::col(u);
      const auto xq = rq.get(u), xk = rk.get(u);
      typename TileQ::vec_t qo, ko;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = sG[j * LDG + c0 + e] - sG[(C / 2 - 1) * LDG + c0 + e];
        qo[e] = to<T>(f32(xq[e]) * __expf(d));
        ko[e] = to<T>(f32(xk[e]) * __expf(-d));
      }
      *reinterpret_cast<typename TileQ::vec_t*>(sQt + j * LDQ + c0) = qo;
      *reinterpret_cast<typename TileQ::vec_t*>(sKt + j * LDQ + c0) = ko;
    }
  }
  lds_barrier();
#pragma unroll
  for (int J = 0; J < 4; ++J) {
    if (J % HW != hh) continue;  // the stripe's other wave takes it
    f32x4 acc = zero4();
    if (J <= sw) tile_mma<T, DK>(acc, sQt + 16 * sw * LDQ, LDQ, sKt + 16 * J * LDQ, LDQ);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r, jj = 16 * J + c16;
      sAqkT[jj * LDT + i] = to<T>((J <= sw && jj <= i) ? a.scale * acc[r] : 0.f);
    }
  }
  lds_barrier();

  // ---- phase 2: loop over value slices
  // X1 = dO S_r diag(e^{b_m}), X2 = V dS_{r+1} diag(e^{b_C - b_m}), Adv = dO V^T
  // (this wave's key-channel tiles ct0 .. ct0 + NTW - 1 and dO V^T tiles J % HW = hh)
  f32x4 X1[NTW], X2[NTW], Adv[4];
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) { X1[ct] = zero4(); X2[ct] = zero4(); }
#pragma unroll
  for (int J = 0; J < 4; ++J) Adv[J] = zero4();
  T* dvrow = static_cast<T*>(a.dv_out) + tok_off(b, r0, h, a.T, a.H, a.dv);
  // every value slice's global operands are requested one slice ahead
  typedef T v8 __attribute__((ext_vector_type(8)));
  constexpr int NPS = BV * DK / 8 / NT;  // 8-element pieces of S_r (and dS) per thread
  static_assert(NPS >= 1 && BV * DK / 8 % NT == 0, "piece split");
  struct Slice {
    v8 s[NPS], d[NPS];
    RowTile<T, BV, NT> rv, rdo;
  };
  auto load_slice = [&](Slice& sl, int vv0) {
#pragma unroll
    for (int p = 0; p < NPS; ++p) {
      const int idx = tid + p * NT, row = idx / (DK / 8), c0 = (idx % (DK / 8)) * 8;
      sl.s[p] = *reinterpret_cast<const v8*>(Sst + (size_t)(vv0 + row) * DK + c0);
      sl.d[p] = *reinterpret_cast<const v8*>(dSst + (size_t)(vv0 + row) * DK + c0);
    }
    sl.rv.load(v + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
    sl.rdo.load(dO + tok_off(b, r0, h, a.T, a.H, a.dv) + vv0, gsv, nrow);
  };
  Slice cur;
  load_slice(cur, 0);
  // sum_v S_r[c][v] dS_{r+1}[c][v] for this thread's 8 channels (every piece
  // of a thread covers the same channels)
  static_assert(NT % (DK / 8) == 0, "channels per thread");
  float rdot[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) rdot[e] = 0.f;
  for (int vv0 = 0; vv0 < a.dv; vv0 += BV) {
    // states, rows v: S_r diag(e^{b_m}) and dS_{r+1} diag(e^{b_C - b_m}); the
    // products over v read them with transposing LDS reads
#pragma unroll
    for (int p = 0; p < NPS; ++p) {
      const int idx = tid + p * NT, row = idx / (DK / 8), c0 = (idx % (DK / 8)) * 8;
      v8 s_scaled, ds_scaled;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        s_scaled[e] = to<T>(f32(cur.s[p][e]) * sBm[c0 + e]);
        ds_scaled[e] = to<T>(f32(cur.d[p][e]) * sBCm[c0 + e]);
        rdot[e] += f32(cur.s[p][e]) * f32(cur.d[p][e]);
      }
      *reinterpret_cast<v8*>(sS + row * LDQ + c0) = s_scaled;
      *reinterpret_cast<v8*>(sdS + row * LDQ + c0) = ds_scaled;
    }
    cur.rv.store(sV, LDV);
    cur.rdo.store(sdO, LDV);
    if (vv0 + BV < a.dv) load_slice(cur, vv0 + BV);
    lds_barrier();
#pragma unroll
    for (int k0 = 0; k0 < BV; k0 += 32) {
      const Frag<T> fo = ld_frag(sdO + 16 * sw * LDV + k0, LDV);
      const Frag<T> fv = ld_frag(sV + 16 * sw * LDV + k0, LDV);
#pragma unroll
      for (int ct = 0; ct < NTW; ++ct) {
        mma(X1[ct], fo, ld_frag_tr(sS + k0 * LDQ + 16 * (ct0 + ct), LDQ));
        mma(X2[ct], fv, ld_frag_tr(sdS + k0 * LDQ + 16 * (ct0 + ct), LDQ));
      }
    }
#pragma unroll
    for (int J = 0; J < 4; ++J)
      if (J <= sw && J % HW == hh) tile_mma<T, BV>(Adv[J], sdO + 16 * sw * LDV, LDV, sV + 16 * J * LDV, LDV);
    // dv = s (Qt Kt^T masked)^T dO + Kt (dS e^{b_C - b_m})^T  for rows of stripe sw
#pragma unroll
    for (int tq = 0; tq < BV / 16 / HW; ++tq) {
      const int tn = HW * tq + hh;
      f32x4 acc = zero4();
      tile_mma_bt<T, C>(acc, sAqkT + 16 * sw * LDT, LDT, sdO + 16 * tn, LDV);
      tile_mma<T, DK>(acc, sKt + 16 * sw * LDQ, LDQ, sdS + 16 * tn * LDQ, LDQ);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int jr = 16 * sw + 4 * g4 + r;
        if (jr < nrow) dvrow[jr * gsv + vv0 + 16 * tn + c16] = to<T>(acc[r]);
      }
    }
    lds_barrier();
  }

  // ---- phase 3: intra terms with A_dv[t][j] = dO_t . v_j (j <= t)
#pragma unroll
  for (int J = 0; J < 4; ++J) {
    if (J % HW != hh) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r, jj = 16 * J + c16;
      sAdv[i * LDT + jj] = to<T>((J <= sw && jj <= i) ? Adv[J][r] : 0.f);
    }
  }
  lds_barrier();
  f32x4 Y2[NTW];
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) {
    tile_mma_bt<T, C>(X1[ct], sAdv + 16 * sw * LDT, LDT, sKt + 16 * (ct0 + ct), LDQ);
    Y2[ct] = zero4();
    tile_mma_tr<T, C>(Y2[ct], sAdv + 16 * sw, LDT, sQt + 16 * (ct0 + ct), LDQ);
  }
  lds_barrier();  // sAdv dead: sTot may reuse the region

  // ---- phase 4: epilogue per element (row i of stripe sw, key channel c)
  // every global operand of the epilogue requested at once (rows clamped into
  // the sequence), then the per-element arithmetic
  const size_t rowoff = tok_off(b, r0, h, a.T, a.H, DK);
  T* dqc_io = static_cast<T*>(a.dqc_io) + rowoff;
  float* dqc_f = a.dqc + rowoff;
  float* dkg_f = a.dk_gla + rowoff;
  float* db_f = a.db + rowoff;
  float qv[NTW][4], kv[NTW][4], cv[NTW][4];
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      const int off = (i < nrow ? i : nrow - 1) * (int)gsk + 16 * (ct0 + ct) + c16;
      qv[ct][r] = f32(qc[rowoff + off]);
      kv[ct][r] = f32(k[rowoff + off]);
      cv[ct][r] = a.corr[rowoff + off];
    }
  float kdk[NTW];  // sum over the chunk's rows of k * dk^inter
  float dl[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) {
    kdk[ct] = 0.f;
    const int c = 16 * (ct0 + ct) + c16;
    const float bm = sG[(C / 2 - 1) * LDG + c];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      if (i < nrow) {
        const float d = sG[i * LDG + c] - bm;
        const float dqc = a.scale * __expf(d) * X1[ct][r];
        const float inter = __expf(-d) * X2[ct][r];
        const float dkg = __expf(-d) * (Y2[ct][r] * a.scale) + inter;
        const int off = i * (int)gsk + c;
        const float db = qv[ct][r] * dqc - kv[ct][r] * dkg;
        dqc_f[off] = dqc;
        dqc_io[off] = to<T>(dqc);
        dkg_f[off] = dkg;
        db_f[off] = db;
        kdk[ct] += kv[ct][r] * inter;
        dl[r] -= dqc * cv[ct][r];
      }
    }
  }
  // dlam: this wave's channels summed over the 16-lane row group, then (two
  // waves per stripe) the second half's share added through LDS
#pragma unroll
  for (int r = 0; r < 4; ++r) dl[r] = row16_sum(dl[r]);
  if constexpr (HW > 1) {
    if (hh == 1 && c16 == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) sDl[16 * sw + 4 * g4 + r] = dl[r];
    lds_barrier();
    if (hh == 0)
#pragma unroll
      for (int r = 0; r < 4; ++r) dl[r] += sDl[16 * sw + 4 * g4 + r];
  }
  if (hh == 0)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * sw + 4 * g4 + r;
      if (c16 == 0 && i < nrow) a.dlam[((size_t)b * a.T + r0 + i) * a.H + h] = dl[r];
    }
  // decay gradient at the next chunk's first token:
  //   e^{b_C} sum_v S_r dS_{r+1} + sum_j k_j * dk_j^inter
  // (zero after the last chunk, where dS_{r+1} = 0); wave sums in a fixed order
  float* sRow = sTot + 4 * DK;
#pragma unroll
  for (int ct = 0; ct < NTW; ++ct) {
    float x = kdk[ct];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if (g4 == 0) sTot[sw * DK + 16 * (ct0 + ct) + c16] = x;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float x = rdot[e];
#pragma unroll
    for (int m = DK / 8; m < 64; m *= 2) x += __shfl_xor(x, m);
    rdot[e] = x;
  }
  if (l < DK / 8)
#pragma unroll
    for (int e = 0; e < 8; ++e) sRow[w * DK + 8 * l + e] = rdot[e];
  lds_barrier();
  if (tid < DK) {
    const float kd = sTot[tid] + sTot[DK + tid] + sTot[2 * DK + tid] + sTot[3 * DK + tid];
    float sd = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) sd += sRow[ww * DK + tid];
    a.dg_next[((size_t)bh * N + ci) * DK + tid] = __expf(sG[(C - 1) * LDG + tid]) * sd + kd;
  }
}

// ----------------------------------------------------------------------------
// dg_t = sum_{s >= t} db_s: one workgroup per chunk, one thread per channel;
// the rows of the chunk are summed here and the later chunks enter through the
// decay gradient at the next chunk's first token (dg_next).
template <typename TG>
__global__ __launch_bounds__(kThreads) void gla_dg_kernel(const DgArgs a) {
  constexpr int C = kChunk, HC = C / 2;
  __shared__ float sHalf[kThreads];
  const int N = (a.T + C - 1) / C;
  const int lb = blockIdx.x;
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const int r0 = ci * C;
  const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
  const int hd = a.H * a.dk;
  TG* dg = static_cast<TG*>(a.dg) + tok_off(b, r0, h, a.T, a.H, a.dk);
  const float* db = a.db + tok_off(b, r0, h, a.T, a.H, a.dk);
  // thread (c, half): half 1 takes rows 32..63 of channel c, half 0 rows 0..31
  const int npc = kThreads / 2;  // channels per pass
  for (int c0 = 0; c0 < a.dk; c0 += npc) {
    const int c = c0 + (threadIdx.x % npc), half = threadIdx.x / npc;
    const bool on = c < a.dk;
    // sum over the later chunks (half 1 only)
    const float later = (on && half == 1) ? a.dg_next[((size_t)bh * N + ci) * a.dk + c] : 0.f;
    float x[HC];
#pragma unroll
    for (int j = 0; j < HC; ++j) {
      const int row = HC * half + j;
      x[j] = on ? db[(row < nrow ? row : nrow - 1) * hd + c] : 0.f;
    }
    float run = 0.f;  // sum of this half's rows
#pragma unroll
    for (int j = 0; j < HC; ++j) run += (HC * half + j < nrow) ? x[j] : 0.f;
    sHalf[threadIdx.x] = run + later;
    __syncthreads();
    // half 0 starts from everything after row 31; half 1 from the later chunks
    float acc = half == 0 ? sHalf[threadIdx.x + npc] : later;
    __syncthreads();
#pragma unroll
    for (int j = HC - 1; j >= 0; --j) {
      const int row = HC * half + j;
      if (on && row < nrow) {
        acc += x[j];
        dg[row * hd + c] = static_cast<TG>(acc);
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Key gradient of the contraction, dk_j = H_j k_j + D_j + (within-chunk terms),
// with the suffix sums over later tokens
//   H_j = sum_{t > chunk of j} rho_t (u_t q_t^T + q_t u_t^T),  rho_t = -lam_t / t,
//   D_j = sum_{t > chunk of j} (lam_t/t^2) (u_t (m_t.q_t) + q_t (m_t.u_t)).
// Both are plain (undecayed) sums, so the chunks are cut into segments of
// `seg`: ccq_dk_stats_kernel forms every segment's H and D and every chunk's
// D (one workgroup per segment, all segments in parallel), and
// ccq_dk_kernel starts each segment from the sum over the later segments and
// walks the segment's chunks from last to first.  For large DK the 16 x 16
// tiles of H (and the output columns of ccq_dk_kernel) are split over NSPLIT
// workgroups per segment; each stages the whole chunk.
// Both kernels stage q and rho u as row-major chunk tiles (16-byte writes) and
// read them feature-major with transposing reads where a product runs over the
// chunk's rows.
template <typename T, int DK, int NSPLIT, int NWV>
__global__ __launch_bounds__(64 * NWV, 1) void ccq_dk_stats_kernel(const CcqDkArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P;
  constexpr int NTHR = 64 * NWV;
  constexpr int NT16 = DK / 16, NPW = NT16 * NT16 / (NWV * NSPLIT);
  constexpr int NPART = NTHR / DK;
  static_assert(NPW >= 1 && NTHR % DK == 0, "tile split");
  // row-major staging with coalesced loads (adjacent lanes along a row)
  typedef RowTile<T, DK, NTHR> Tile;

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sRU[C * LDQ];  // rho u
  __shared__ float sA[C], sB[C];            // -(m.q)/t and -rho (m.u)/t
  __shared__ float sDp[NTHR];

  const int N = (a.T + C - 1) / C;
  const int NS = (N + a.seg - 1) / a.seg;
  // the NSPLIT workgroups of a segment are consecutive logical blocks: one
  // XCD (one L2) at about the same time, so each chunk comes from HBM once
  const int lbs = xcd_logical_block(blockIdx.x, gridDim.x);
  const int split = lbs % NSPLIT, lb = lbs / NSPLIT;  // split: this workgroup's share of the tiles
  const int bh = lb / NS, sg = lb % NS;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const int tw0 = (split * NWV + w) * NPW;  // first tile of this wave
  const T* q = static_cast<const T*>(a.q);
  const T* uu = static_cast<const T*>(a.u);
  const size_t gs = (size_t)a.H * DK;
  const int c_begin = sg * a.seg;
  const int c_end = (c_begin + a.seg) < N ? (c_begin + a.seg) : N;

  f32x4 H[NPW];
#pragma unroll
  for (int u = 0; u < NPW; ++u) H[u] = zero4();
  float dsum = 0.f;

  Tile rq, ru;
  RowScales<Tile> fl;         // lambda of each staged vector's row
  RowScalar rlam, rmq, rmu;   // wave 0: lane = row
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    rq.load(q + tok_off(b, r0, h, a.T, a.H, DK), gs, nrow);
    ru.load(uu + tok_off(b, r0, h, a.T, a.H, DK), gs, nrow);
    const size_t t0i = ((size_t)b * a.T + r0) * a.H + h;
    fl.load(a.lam + t0i, (size_t)a.H, nrow);
    if (w == 0) {
      rlam.load(a.lam + t0i, (size_t)a.H, l, nrow);
      rmq.load(a.mdot_q + t0i, (size_t)a.H, l, nrow);
      rmu.load(a.mdot_u + t0i, (size_t)a.H, l, nrow);
    }
  };
  if (c_begin < c_end) prefetch(c_begin);

  for (int ci = c_begin; ci < c_end; ++ci) {
    lds_barrier();
    {
      if (w == 0) {
        const float tpos = (float)(ci * C + l + 1);
        const float rho = -rlam.get() / tpos;
        sA[l] = a.centered ? -rmq.get() / tpos : 0.f;
        sB[l] = a.centered ? -rho * rmu.get() / tpos : 0.f;
      }
      rq.store(sQ, LDQ);
#pragma unroll
      for (int u = 0; u < Tile::NV; ++u) {
        if (!Tile::mine(u)) continue;
        const int j = Tile::row(u);
        const float rho = -fl.f[u] / (float)(ci * C + j + 1);
        const auto x = ru.get(u);
        typename Tile::vec_t y;
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = to<T>(rho * f32(x[e]));
        *reinterpret_cast<typename Tile::vec_t*>(sRU + j * LDQ + Tile::col(u)) = y;
      }
    }
    if (ci + 1 < c_end) prefetch(ci + 1);
    lds_barrier();
#pragma unroll
    for (int u = 0; u < NPW; ++u) {
      const int tau = tw0 + u, tr = tau / NT16, tc = tau % NT16;
      tile_mma_tr<T, C>(H[u], sRU + 16 * tr, LDQ, sQ + 16 * tc, LDQ);
      tile_mma_tr<T, C>(H[u], sQ + 16 * tr, LDQ, sRU + 16 * tc, LDQ);
    }
    if (split == 0) {  // this chunk's mean-term vector, NPART threads per key channel
      const int n = tid % DK, part = tid / DK;
      float x = 0.f;
#pragma unroll 8
      for (int t = part * (C / NPART); t < (part + 1) * (C / NPART); ++t)
        x += sA[t] * f32(sRU[t * LDQ + n]) + sB[t] * f32(sQ[t * LDQ + n]);
      sDp[tid] = x;
    }
    lds_barrier();
    if (split == 0 && tid < DK) {
      float x = sDp[tid];
#pragma unroll
      for (int p2 = 1; p2 < NPART; ++p2) x += sDp[p2 * DK + tid];
      a.dchunk[((size_t)bh * N + ci) * DK + tid] = x;
      dsum += x;
    }
  }
  float* hs = a.hseg + ((size_t)bh * NS + sg) * DK * DK;
#pragma unroll
  for (int u = 0; u < NPW; ++u) {
    const int tau = tw0 + u, tr = tau / NT16, tc = tau % NT16;
#pragma unroll
    for (int r = 0; r < 4; ++r) hs[(size_t)(16 * tr + 4 * g4 + r) * DK + 16 * tc + c16] = H[u][r];
  }
  if (split == 0 && tid < DK) a.dseg[((size_t)bh * NS + sg) * DK + tid] = dsum;
}

// In place, per head: segment s's H and D become the sums over the later
// segments s' > s (exclusive suffix sums), four elements per thread.
__global__ __launch_bounds__(kThreads) void ccq_dk_suffix_kernel(const CcqDkArgs a) {
  const int N = (a.T + kChunk - 1) / kChunk;
  const int NS = (N + a.seg - 1) / a.seg;
  const size_t per = (size_t)a.dk * a.dk + a.dk;  // H and D elements of one segment
  const size_t i4 = ((size_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  const int bh = blockIdx.y;
  if (i4 >= per) return;
  const bool isH = i4 < (size_t)a.dk * a.dk;
  float* base = isH ? a.hseg + (size_t)bh * NS * a.dk * a.dk + i4
                    : a.dseg + (size_t)bh * NS * a.dk + (i4 - (size_t)a.dk * a.dk);
  const size_t stride = isH ? (size_t)a.dk * a.dk : (size_t)a.dk;
  f32x4 acc = zero4();
  for (int s2 = NS - 1; s2 >= 0; --s2) {
    f32x4* p = reinterpret_cast<f32x4*>(base + s2 * stride);
    const f32x4 x = *p;
    *p = acc;
    acc += x;
  }
}

// Reverse walk over one segment's chunks per (head, segment).  Wave w owns
// NTW 16-wide tiles of output columns n and keeps, in MFMA accumulators, the
// carried H[c][n] for every c (H is symmetric, so these columns are also its
// rows) and, in registers, D[n]; both start from the sums over the later
// segments.  Per chunk, with j <= t:
//   W1[t][j] = q_t . k_j - (m_t.q_t)/t            applied to rho_t u_t
//   W2[t][j] = rho_t (u_t . k_j - (m_t.u_t)/t)     applied to q_t
//   dk_j = H k_j + D + sum_{t>=j} (W1[t][j] rho_t u_t + W2[t][j] q_t),
// then H += sum_t rho_t (u_t q_t^T + q_t u_t^T) and D += the chunk's D.  For
// bf16, H and the weights W enter the products as a bf16 head plus a bf16 tail.
// The output columns are split over NSPLIT workgroups per segment.
// W2 is formed from the staged rho u (rho_t u_t . k_j - rho_t (m_t.u_t)/t).
template <typename T, int DK, int NSPLIT, int NWV>
__global__ __launch_bounds__(64 * NWV, 1) void ccq_dk_kernel(const CcqDkArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr bool kSplit = sizeof(T) == 2;
  constexpr int LDQ = DK + P, LDA = C + P;
  constexpr int NCT = DK / 16;  // 16-row tiles of the contraction index c
  constexpr int NTHR = 64 * NWV;
  constexpr int NTW = DK / (16 * NWV * NSPLIT);  // output column tiles per wave
  // row-major staging with coalesced loads (adjacent lanes along a row)
  typedef RowTile<T, DK, NTHR> Tile;
  constexpr int NK = DK / 32;
  static_assert(NTW >= 1, "column split");

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sRU[C * LDQ];  // rho u
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sW1h[C * LDA];   // transposed: [j][t]
  __shared__ __align__(16) T sW1l[kSplit ? C * LDA : 8];
  __shared__ __align__(16) T sW2h[C * LDA];
  __shared__ __align__(16) T sW2l[kSplit ? C * LDA : 8];
  __shared__ float sRho[C], sMq[C], sMu[C];

  const int N = (a.T + C - 1) / C;
  const int NS = (N + a.seg - 1) / a.seg;
  // the NSPLIT workgroups of a segment are consecutive logical blocks (one L2)
  const int lbs = xcd_logical_block(blockIdx.x, gridDim.x);
  const int split = lbs % NSPLIT, lb = lbs / NSPLIT;
  const int bh = lb / NS, sg = lb % NS;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const int nt0 = (split * NWV + w) * NTW;  // first output column tile of this wave
  const T* q = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  const T* uu = static_cast<const T*>(a.u);
  T* dk_out = static_cast<T*>(a.dk_out);
  const size_t gs = (size_t)a.H * DK;
  const int c_begin = sg * a.seg;
  const int c_end = (c_begin + a.seg) < N ? (c_begin + a.seg) : N;

  // the weights' tiles above the diagonal stay zero
  for (int idx = tid; idx < C * LDA; idx += NTHR) {
    sW1h[idx] = to<T>(0.f);
    sW2h[idx] = to<T>(0.f);
    if constexpr (kSplit) {
      sW1l[idx] = to<T>(0.f);
      sW2l[idx] = to<T>(0.f);
    }
  }

  // the sums over the later segments (suffix sums formed by ccq_dk_suffix_kernel)
  f32x4 Hc[NCT][NTW];
  float dreg[NTW];
#pragma unroll
  for (int x = 0; x < NTW; ++x) {
    dreg[x] = 0.f;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) Hc[ct][x] = zero4();
  }
  {  // H[c][n] = H[n][c] (H is symmetric): four consecutive c per load
    const float* hs = a.hseg + ((size_t)bh * NS + sg) * DK * DK;
#pragma unroll
    for (int x = 0; x < NTW; ++x) {
      const int n = 16 * (nt0 + x) + c16;
      dreg[x] = a.dseg[((size_t)bh * NS + sg) * DK + n];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
        Hc[ct][x] = *reinterpret_cast<const f32x4*>(hs + (size_t)n * DK + 16 * ct + 4 * g4);
    }
  }

  Tile rq, ru, rk;
  RowScales<Tile> fl;         // lambda of each staged vector's row
  RowScalar rlam, rmq, rmu;   // wave 0: lane = row
  auto prefetch = [&](int ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    // (at DK = 256 with the row offsets formed at the loads: fewer registers
    // held across the chunk loop, less spill; measured 437 -> 426 us there,
    // slightly slower at DK = 128)
    auto ld = [&](Tile& t, const T* src) {
      if constexpr (DK >= 256) t.load_opaque(src, gs, nrow);
      else t.load(src, gs, nrow);
    };
    ld(rq, q + tok_off(b, r0, h, a.T, a.H, DK));
    ld(ru, uu + tok_off(b, r0, h, a.T, a.H, DK));
    ld(rk, k + tok_off(b, r0, h, a.T, a.H, DK));
    const size_t t0i = ((size_t)b * a.T + r0) * a.H + h;
    fl.load(a.lam + t0i, (size_t)a.H, nrow);
    if (w == 0) {
      rlam.load(a.lam + t0i, (size_t)a.H, l, nrow);
      rmq.load(a.mdot_q + t0i, (size_t)a.H, l, nrow);
      rmu.load(a.mdot_u + t0i, (size_t)a.H, l, nrow);
    }
  };
  if (c_begin < c_end) prefetch(c_end - 1);

  for (int ci = c_end - 1; ci >= c_begin; --ci) {
    const int r0 = ci * C;
    const int nrow = (a.T - r0) < C ? (a.T - r0) : C;
    lds_barrier();  // (A)
    {
      if (w == 0) {
        const float tpos = (float)(r0 + l + 1);
        sRho[l] = -rlam.get() / tpos;
        sMq[l] = a.centered ? rmq.get() / tpos : 0.f;
        sMu[l] = a.centered ? rmu.get() / tpos : 0.f;
      }
      rq.store(sQ, LDQ);
      rk.store(sK, LDQ);
#pragma unroll
      for (int u = 0; u < Tile::NV; ++u) {
        if (!Tile::mine(u)) continue;
        const int j = Tile::row(u);
        const float rho = -fl.f[u] / (float)(r0 + j + 1);
        const auto x = ru.get(u);
        typename Tile::vec_t y;
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = to<T>(rho * f32(x[e]));
        *reinterpret_cast<typename Tile::vec_t*>(sRU + j * LDQ + Tile::col(u)) = y;
      }
    }
    float dcv[NTW];  // this chunk's D, added after its outputs
#pragma unroll
    for (int x = 0; x < NTW; ++x) dcv[x] = a.dchunk[((size_t)bh * N + ci) * DK + 16 * (nt0 + x) + c16];
    // the backbone's part of dk for this wave's outputs, requested before the
    // products: here at DK = 256 (fewer registers live in the dk-row products),
    // else at the start of those products (measured faster there)
    const size_t rowoff = tok_off(b, r0, h, a.T, a.H, DK);
    constexpr bool kEarlyDkg = DK >= 256;
    float dkg[NTW][4][4];
    auto load_dkg = [&](int x) {
#pragma unroll
      for (int J = 0; J < 4; ++J)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int jr = 16 * J + 4 * g4 + r;
          dkg[x][J][r] = a.dk_gla[rowoff + (jr < nrow ? jr : nrow - 1) * (int)gs + 16 * (nt0 + x) + c16];
        }
    };
    if constexpr (kEarlyDkg)
#pragma unroll
      for (int x = 0; x < NTW; ++x) load_dkg(x);
    if (ci > c_begin) prefetch(ci - 1);
    lds_barrier();  // (B)

    // intra weights: the ten tiles on or below the diagonal, over the waves
#pragma unroll
    for (int s3 = 0; s3 < (10 + NWV - 1) / NWV; ++s3) {
      const int t = w + NWV * s3;
      if (t < 10) {
        const int I = intra_tile_row(t), J = intra_tile_col(t);
        f32x4 s1 = zero4(), s2 = zero4();  // q . k and (rho u) . k
#pragma unroll
        for (int k0 = 0; k0 < DK; k0 += 32) {
          const Frag<T> kf = ld_frag(sK + 16 * J * LDQ + k0, LDQ);
          mma(s1, ld_frag(sQ + 16 * I * LDQ + k0, LDQ), kf);
          mma(s2, ld_frag(sRU + 16 * I * LDQ + k0, LDQ), kf);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tt = 16 * I + 4 * g4 + r, jj = 16 * J + c16;
          const bool on = jj <= tt;
          const float w1 = on ? s1[r] - sMq[tt] : 0.f;
          const float w2 = on ? s2[r] - sRho[tt] * sMu[tt] : 0.f;
          if constexpr (kSplit) {
            bf16_t hi, lo;
            split_bf16(w1, hi, lo);
            sW1h[jj * LDA + tt] = hi;
            sW1l[jj * LDA + tt] = lo;
            split_bf16(w2, hi, lo);
            sW2h[jj * LDA + tt] = hi;
            sW2l[jj * LDA + tt] = lo;
          } else {
            sW1h[jj * LDA + tt] = w1;
            sW2h[jj * LDA + tt] = w2;
          }
        }
      }
    }
    lds_barrier();  // (C)

    // dk rows j (all four row tiles), this wave's columns n.  H enters one k
    // step at a time (its bf16 head and tail formed just before use), the four
    // row tiles accumulating side by side: each tile sums the same products in
    // the same order as a tile-by-tile walk, with a quarter of the registers.
#pragma unroll
    for (int x = 0; x < NTW; ++x) {
      const int nt = nt0 + x;
      if constexpr (!kEarlyDkg) load_dkg(x);
      f32x4 acc[4];
#pragma unroll
      for (int J = 0; J < 4; ++J) acc[J] = zero4();
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        Frag<T> hh, hl;
        if constexpr (kSplit) {
          const f32x4 p0 = Hc[2 * m][x], p1 = Hc[2 * m + 1][x];
          hh = acc_pair_frag<T>(p0, p1);
          f32x4 r0v, r1v;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            r0v[e] = p0[e] - f32(hh.v[e]);
            r1v[e] = p1[e] - f32(hh.v[4 + e]);
          }
          hl = acc_pair_frag<T>(r0v, r1v);
        } else {
          hh = acc_pair_frag<T>(Hc[2 * m][x], Hc[2 * m + 1][x]);
        }
#pragma unroll
        for (int J = 0; J < 4; ++J) {
          const Frag<T> kf = ld_frag_acc(sK + 16 * J * LDQ + 32 * m, (size_t)LDQ);
          mma(acc[J], kf, hh);
          if constexpr (kSplit) mma(acc[J], kf, hl);
        }
      }
      Frag<T> f1[2], f2[2];
#pragma unroll
      for (int m2 = 0; m2 < 2; ++m2) {
        f1[m2] = ld_frag_tr(sRU + 32 * m2 * LDQ + 16 * nt, LDQ);
        f2[m2] = ld_frag_tr(sQ + 32 * m2 * LDQ + 16 * nt, LDQ);
      }
#pragma unroll
      for (int J = 0; J < 4; ++J) {
#pragma unroll
        for (int m2 = 0; m2 < 2; ++m2) {
          mma(acc[J], ld_frag(sW1h + 16 * J * LDA + 32 * m2, LDA), f1[m2]);
          mma(acc[J], ld_frag(sW2h + 16 * J * LDA + 32 * m2, LDA), f2[m2]);
          if constexpr (kSplit) {
            mma(acc[J], ld_frag(sW1l + 16 * J * LDA + 32 * m2, LDA), f1[m2]);
            mma(acc[J], ld_frag(sW2l + 16 * J * LDA + 32 * m2, LDA), f2[m2]);
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int jr = 16 * J + 4 * g4 + r;
          if (jr < nrow) {
            dk_out[rowoff + jr * (int)gs + 16 * nt + c16] = to<T>(dkg[x][J][r] + acc[J][r] + dreg[x]);
          }
        }
      }
    }

    // H += (rho u)^T q + q^T (rho u) for this wave's columns; D += this chunk's D
    Frag<T> bq[NTW][2], bu[NTW][2];
#pragma unroll
    for (int x = 0; x < NTW; ++x)
#pragma unroll
      for (int m2 = 0; m2 < 2; ++m2) {
        bq[x][m2] = ld_frag_tr(sQ + 32 * m2 * LDQ + 16 * (nt0 + x), LDQ);
        bu[x][m2] = ld_frag_tr(sRU + 32 * m2 * LDQ + 16 * (nt0 + x), LDQ);
      }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int m2 = 0; m2 < 2; ++m2) {
        const Frag<T> au = ld_frag_tr(sRU + 32 * m2 * LDQ + 16 * ct, LDQ);
        const Frag<T> aq = ld_frag_tr(sQ + 32 * m2 * LDQ + 16 * ct, LDQ);
#pragma unroll
        for (int x = 0; x < NTW; ++x) {
          mma(Hc[ct][x], au, bq[x][m2]);
          mma(Hc[ct][x], aq, bu[x][m2]);
        }
      }
#pragma unroll
    for (int x = 0; x < NTW; ++x) dreg[x] += dcv[x];
  }
}

// ----------------------------------------------------------------------------
namespace {
template <typename T, typename TG, int DK, int BV, int NW = 4>
hipError_t run_bwd_chunk(const GlaBwdArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * ((a.T + kChunk - 1) / kChunk);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_bwd_chunk_kernel<T, TG, DK, BV, NW>), dim3(nblk), dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_ccq_dk(const CcqDkArgs& a, hipStream_t st) {
  const int N = (a.T + kChunk - 1) / kChunk;
  if (a.seg <= 0) return hipErrorInvalidValue;
  const int NS = (N + a.seg - 1) / a.seg;
  const int nseg = a.B * a.H * NS;
  if (nseg == 0) return hipSuccess;
  // eight waves per workgroup (two per SIMD) for ccq_dk_kernel from DK = 128
  // and ccq_dk_stats_kernel at DK = 256 (measured: at DK = 128 the statistics
  // run faster with four); at DK = 256 H's tiles (ccq_dk_stats_kernel) and the
  // output columns (ccq_dk_kernel, each wave carrying one 16-column tile of H)
  // are split over two workgroups per segment, so that a wave's share of H
  // fits its registers
  constexpr int NSPLIT_S = DK >= 256 ? 2 : 1, NSPLIT = DK >= 256 ? 2 : 1;
  constexpr int NWV_S = DK >= 256 ? 8 : 4, NWV = DK >= 128 ? 8 : 4;
  hipLaunchKernelGGL((ccq_dk_stats_kernel<T, DK, NSPLIT_S, NWV_S>), dim3(nseg * NSPLIT_S), dim3(64 * NWV_S), 0, st,
                     a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t per4 = ((size_t)DK * DK + DK) / 4;
  hipLaunchKernelGGL(ccq_dk_suffix_kernel, dim3((unsigned)((per4 + kThreads - 1) / kThreads), a.B * a.H),
                     dim3(kThreads), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((ccq_dk_kernel<T, DK, NSPLIT, NWV>), dim3(nseg * NSPLIT), dim3(64 * NWV), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG>
hipError_t chunk_dispatch(const GlaBwdArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (a.dk == 64) return run_bwd_chunk<T, TG, 64, 32>(a, st);
    // eight waves (two per SIMD: the kernel takes a compute unit's LDS) and
    // 64-wide value slices at dk = 128
    if (a.dk == 128) return run_bwd_chunk<T, TG, 128, 64, 8>(a, st);
  } else {
    if (a.dk == 64) return run_bwd_chunk<T, TG, 64, 32>(a, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

bool bwd_supported(int dk, int dv, bool is_bf16, bool gdn) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  if (is_bf16) return dv_ok && (dk == 64 || dk == 128 || (gdn && dk == 256));
  return dv_ok && dk == 64;
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
    if (a.dk == 64) return run_ccq_dk<bf16_t, 64>(a, st);
    if (a.dk == 128) return run_ccq_dk<bf16_t, 128>(a, st);
    if (a.dk == 256) return run_ccq_dk<bf16_t, 256>(a, st);
  } else {
    if (a.dk == 64) return run_ccq_dk<float, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace ccq
