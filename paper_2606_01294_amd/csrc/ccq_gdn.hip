// ccq_gdn.hip -- Gated DeltaNet backbone chunk forward reading the cleaned queries.
//
// Gated DeltaNet (the cited backbone): S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T)
// + beta_t v_t k_t^T.  Writing S_t = alpha_t S_{t-1} + u_t k_t^T with
// u_t = beta_t (v_t - alpha_t S_{t-1} k_t), and gamma_i = sum_{s<=i} log alpha_s
// inside a chunk entered with state S_r, the rows u_i solve
//
//   (I + A) U = diag(beta) (V - diag(e^gamma) K S_r^T),
//   A_ij = beta_i e^{gamma_i - gamma_j} (k_i . k_j)  (j < i),
//
// so with Tm = (I + A)^{-1}:  U = Tm R,  R = diag(beta) (V - diag(e^gamma) K S_r^T).
// Then
//
//   o_i     = e^{gamma_i} S_r q_i + sum_{j<=i} e^{gamma_i - gamma_j} (k_j . q_i) u_j
//   S_{r+1} = e^{gamma_C} S_r + U^T diag(e^{gamma_C - gamma}) K.
//
// gdn_tri_kernel forms Tm for every chunk in parallel (MFMA block inversion in
// fp32); gdn_state_kernel walks the chunks of one head in order, keeping a
// slice of S in MFMA accumulators, and stores S_r and U for every chunk;
// gdn_out_kernel then forms the outputs of all chunks in parallel.  S_r and
// U^T are stored fragment-native: per 16-row value tile and 32-wide k step a
// contiguous 16 x 32 block, so the state kernel writes and the output kernel
// reads 1 KB per instruction, already in MFMA operand order.  Rows of S_r are
// in natural feature order (the state kernel keeps its accumulator tiles in
// pair order, ld_frag_tr_acc_pair); rows of U^T are in accumulator-pair order
// (acc_pos) over the chunk's tokens.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// Tm = (I + A)^{-1} of one chunk, plus the chunk's decay coefficients
// (gamma_j, beta_j e^{gamma_j}, beta_j, e^{gamma_C - gamma_j}, e^{gamma_C}), so the
// sequential state pass needs no exponentials.
// Blocks of 16: the diagonal blocks are inverted by forward substitution,
// then wave w forms column block w, X_iw = -D_i sum_{m=w}^{i-1} A_im X_mw.
template <typename T, int DK>
__global__ __launch_bounds__(kThreads) void gdn_tri_kernel(const TriArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P;
  constexpr int LDA = C + 4;  // fp32 pitch of A and X
  // K is dead once A is formed: A and X (fp32) then take its space, which lets
  // four workgroups share a compute unit
  constexpr int kKBytes = C * LDQ * (int)sizeof(T), kAXBytes = 2 * C * LDA * 4;
  __shared__ __align__(16) char sKAX[kKBytes > kAXBytes ? kKBytes : kAXBytes];
  T* const sK = reinterpret_cast<T*>(sKAX);
  float* const sA = reinterpret_cast<float*>(sKAX);
  float* const sX = sA + C * LDA;
  __shared__ __align__(16) float sY[4][16 * 17];
  __shared__ __align__(16) float sGam[C], sBeta[C];

  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / N, ci = lb % N;
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  const int r0 = ci * C;
  if (r0 >= sq.len) return;  // past a packed sequence's end
  const int nrow = (sq.len - r0) < C ? (sq.len - r0) : C;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;

  // all global loads first (K, the log decays and beta), one round trip
  RowTile<T, DK> rk;
  RowScales<RowTile<T, DK>> fk;  // raw keys: row scales (l2 normalisation)
  rk.load(static_cast<const T*>(a.k) + seq_off(sq, r0, h, a.H, DK), (size_t)a.H * DK, nrow);
  if (a.rk) fk.load(a.rk + seq_idx(sq, r0, h, a.H), (size_t)a.H, nrow);
  float la = 0.f, bt = 0.f, rkt = 1.f;
  if (tid < C) {
    const size_t ti = seq_idx(sq, r0 + (tid < nrow ? tid : nrow - 1), h, a.H);
    la = a.logalpha[ti];
    bt = a.beta[ti];
    if (a.rk) rkt = a.rk[ti];
  }
  if (a.rk) fk.apply(rk);
  rk.store(sK, LDQ);
  if (tid < C) {
    float x = tid < nrow ? la : 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(x, off);
      if (tid >= off) x += y;
    }
    bt = tid < nrow ? bt : 0.f;
    const float gC = __shfl(x, C - 1);
    sGam[tid] = x;
    sBeta[tid] = bt;
    float* cf = a.gam + ((size_t)bh * N + ci) * 5 * C + tid;
    cf[0] = x;                      // gamma_j
    // (with raw keys the two coefficients that multiply key rows carry the
    // row's l2 normalisation)
    cf[C] = bt * __expf(x) * rkt;   // beta_j e^{gamma_j}
    cf[2 * C] = bt;                 // beta_j
    cf[3 * C] = __expf(gC - x) * rkt;  // e^{gamma_C - gamma_j}
    cf[4 * C] = __expf(gC);         // e^{gamma_C}
  }
  __syncthreads();

  // A (strictly lower): the ten tiles I >= J dealt to the waves in turn (three,
  // three, two, two); written once every wave is done with K (the upper
  // tiles are never read)
  f32x4 acc[3];
#pragma unroll
  for (int s3 = 0; s3 < 3; ++s3) {
    const int t = w + 4 * s3;
    acc[s3] = zero4();
    if (t < 10)
      tile_mma<T, DK>(acc[s3], sK + 16 * intra_tile_row(t) * LDQ, LDQ, sK + 16 * intra_tile_col(t) * LDQ, LDQ);
  }
  __syncthreads();
#pragma unroll
  for (int s3 = 0; s3 < 3; ++s3) {
    const int t = w + 4 * s3;
    if (t >= 10) continue;
    const int I = intra_tile_row(t), J = intra_tile_col(t);
    // the coefficients read whole and every entry formed before the mask is
    // applied as a select (reads under the mask compile to a branch and a wait
    // each); e^{gamma_i - gamma_j} may overflow above the diagonal, where the
    // select discards it
    const f32x4 gi = *reinterpret_cast<const f32x4*>(sGam + 16 * I + 4 * g4);
    const f32x4 bi = *reinterpret_cast<const f32x4*>(sBeta + 16 * I + 4 * g4);
    const float gj = sGam[16 * J + c16];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * I + 4 * g4 + r, j = 16 * J + c16;
      const float v = bi[r] * __expf(gi[r] - gj) * acc[s3][r];
      sA[i * LDA + j] = j < i ? v : 0.f;
    }
  }
  __syncthreads();

  // diagonal blocks: lane l < 16 of wave w solves column l of block w; each
  // row's sum is kept in four partial sums (terms m mod 4), so that x_i waits
  // for one product with x_{i-1} and two additions instead of the whole row
  if (l < 16) {
    float x[16];
    const float* Ab = sA + 16 * w * LDA + 16 * w;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float p[4] = {i == l ? 1.f : 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 0; m < i; ++m) p[m & 3] -= Ab[i * LDA + m] * x[m];
      x[i] = (p[0] + p[1]) + (p[2] + p[3]);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) sX[(16 * w + i) * LDA + 16 * w + l] = x[i];
  }
  // (the blocks above the diagonal are never written: the output selects zero there)
  __syncthreads();

  // off-diagonal blocks of column block w (LDS traffic local to the wave)
  for (int i = w + 1; i < 4; ++i) {
    f32x4 y = zero4();
    for (int m = w; m < i; ++m) mma16_f32(y, sA + 16 * i * LDA + 16 * m, LDA, sX + 16 * m * LDA + 16 * w, LDA);
#pragma unroll
    for (int r = 0; r < 4; ++r) sY[w][(4 * g4 + r) * 17 + c16] = y[r];
    f32x4 x = zero4();
    mma16_f32(x, sX + 16 * i * LDA + 16 * i, LDA, sY[w], 17);
#pragma unroll
    for (int r = 0; r < 4; ++r) sX[(16 * i + 4 * g4 + r) * LDA + 16 * w + c16] = -x[r];
  }
  __syncthreads();

  // Tm rows i, each 32-column block in acc_pos order: positions 8q .. 8q + 7
  // of a row hold logical columns b + 4 (q % 4) .. + 3 and b + 16 + 4 (q % 4)
  // .. + 3 (b = the block's first column), two 16-byte LDS reads per piece
  T* Tout = static_cast<T*>(a.Tm) + ((size_t)bh * N + ci) * C * C;
  for (int idx = tid; idx < C * C / 8; idx += kThreads) {
    const int i = idx / (C / 8), q = idx % (C / 8);
    const int lc = ((8 * q) & ~31) + 4 * (q & 3);
    f32x4 lo = *reinterpret_cast<const f32x4*>(sX + i * LDA + lc);
    f32x4 hi = *reinterpret_cast<const f32x4*>(sX + i * LDA + lc + 16);
    if ((lc >> 4) > (i >> 4)) lo = zero4();  // above the diagonal blocks
    if (((lc + 16) >> 4) > (i >> 4)) hi = zero4();
    store_acc_pair(Tout + i * C + 8 * q, lo, hi);
  }
}

// State recurrence over the chunks of one head.  A workgroup owns NPR value
// slices of 16 (v = v0 + 16 p + ..); each slice is shared by NH waves, wave
// (p, hq) keeping key features c in [hq DK/NH, (hq+1) DK/NH) of S^T[c][v] in
// MFMA accumulators.  Per chunk:
//   S_r -> states;  P = K S_r^T (partial over the wave's features, summed over
//   the NH waves through LDS);  R = diag(beta) (V - diag(e^gamma) P);
//   U = Tm R -> U^T;  S^T <- e^{gamma_C} S^T + K^T diag(e^{gamma_C - gamma}) U.
// Every product takes its S, R or U operand straight from the accumulators of
// the step before (acc_pair_frag).  K, Tm and the V slice are staged through
// double-buffered LDS.  Splitting the features over NH waves shortens the
// chain of dependent products per chunk and puts NH times more waves on the
// chip, which matters because the chunks of a head are strictly sequential.
template <typename T, int DK, int NPR, int NH>
__global__ __launch_bounds__(64 * NPR * NH, 1) void gdn_state_kernel(const GdnArgs a) {
  constexpr int C = kChunk, NW = NPR * NH, NT = 64 * NW, BVS = 16 * NPR;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDT = C + P, LDV = BVS + P;
  constexpr int DKH = DK / NH;     // key features per wave
  constexpr int NCT = DKH / 16;    // key-feature tiles per wave
  constexpr int NKH = DKH / 32;    // 32-wide k steps per wave
  static_assert(NKH >= 1, "key split");

  __shared__ __align__(16) T sK[2][C * LDQ];
  __shared__ __align__(16) T sT[2][C * LDT];
  __shared__ __align__(16) T sV[2][C * LDV];
  __shared__ __align__(16) float sCf[2][4][C];  // beta e^gamma, beta, e^{gamma_C - gamma}, e^{gamma_C}
  __shared__ __align__(16) f32x4 sX[NH > 1 ? NW * 4 * 64 : 1];  // partial P of every wave

  const int nvt = a.dv / BVS;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  // heads in head-major order: the workgroups of consecutive logical blocks
  // (one compute-unit cluster) then hold one head of every sequence, which
  // balances the clusters when a packed batch's sequences differ in length
  const int hm = lb / nvt;
  const int bh = (hm % a.B) * a.H + hm / a.B;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const int pr = w / NH, hq = w % NH;
  const int v0 = (lb % nvt) * BVS;
  const int vs = 16 * pr + c16;     // value column within the workgroup's slice
  const int v = v0 + vs;
  const int c0 = hq * DKH;          // first key feature of this wave
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  const int NL = (sq.len + C - 1) / C;  // chunks walked (a packed sequence's own)
  const T* k = static_cast<const T*>(a.k);
  const T* vin = static_cast<const T*>(a.v);
  const T* Tg = static_cast<const T*>(a.Tm);

  // S^T[c][v] in pair order: c = c0 + pair_feat(tc, g4) + r, so that the
  // packed operand of tiles 2m, 2m + 1 holds 8 consecutive features per lane
  // group (the states are stored so, and K is read with plain 16-byte reads)
  f32x4 S[NCT];
#pragma unroll
  for (int tc = 0; tc < NCT; ++tc) {
    if (a.S0)
      S[tc] = *reinterpret_cast<const f32x4*>(a.S0 + ((size_t)bh * a.dv + v) * DK + c0 + pair_feat(tc, g4));
    else
      S[tc] = zero4();
  }

  // chunk data prefetched into registers one iteration ahead
  struct Stage {
    RowTile<T, DK, NT> rk;
    RowTile<T, C, NT> rt;
    RowTile<T, BVS, NT> rv;
    RowScalar cf[4];
  };
  Stage st;
  auto prefetch = [&](Stage& sg, int ci) {
    const int r0 = ci * C;
    const int nrow = (sq.len - r0) < C ? (sq.len - r0) : C;
    sg.rk.load(k + seq_off(sq, r0, h, a.H, DK), (size_t)a.H * DK, nrow);
    sg.rt.load(Tg + ((size_t)bh * N + ci) * C * C, (size_t)C, C);
    sg.rv.load(vin + seq_off(sq, r0, h, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
    if (tid < C) {
#pragma unroll
      for (int q = 0; q < 4; ++q) sg.cf[q].load(a.gam + (((size_t)bh * N + ci) * 5 + 1 + q) * C, 1, tid, C);
    }
  };

  // S_r and U^T of chunk ci are written back at the start of iteration ci + 1,
  // after that iteration's LDS copies: all vector memory operations share one
  // in-order counter, so a store issued just before the next chunk's loads
  // are waited for would have its write latency added to every chunk.
  // Both are stored fragment-native: 1 KB per (value tile, k step).
  const int vt = (v0 >> 4) + pr;
  T* st_base = static_cast<T*>(a.states) + (((size_t)vt * (DK / 32) + hq * NKH) * 16 + c16) * 32 + 8 * g4;
  T* u_base = static_cast<T*>(a.U) + ((size_t)vt * 2 * 16 + c16) * 32 + 8 * g4;
  Frag<T> sf[NKH], uf[2];
  auto write_back = [&](int cw) {
    T* st_out = st_base + ((size_t)bh * N + cw) * a.dv * DK;
    if (cw % a.sstride == 0)
#pragma unroll
      for (int m = 0; m < NKH; ++m) store_frag(st_out + 16 * 32 * m, sf[m]);
    if (hq == 0) {
      T* u_out = u_base + ((size_t)bh * N + cw) * a.dv * C;
      store_frag(u_out, uf[0]);
      store_frag(u_out + 16 * 32, uf[1]);
    }
  };

  auto step = [&](Stage& sg, int ci) {
    const int buf = ci & 1;
    // the LDS buffer was released by every wave at the previous barrier
    sg.rk.store(sK[buf], LDQ);
    sg.rt.store(sT[buf], LDT);
    sg.rv.store(sV[buf], LDV);
    if (tid < C) {
#pragma unroll
      for (int q = 0; q < 4; ++q) sCf[buf][q][tid] = sg.cf[q].get();
    }
    if (ci > 0) write_back(ci - 1);
    if (ci + 1 < NL) prefetch(sg, ci + 1);
    // the barriers of the step order LDS only: a __syncthreads() fence would
    // wait for the prefetch just issued and for the stores
    lds_barrier();
    const T* Kb = sK[buf];

    // P = K S_r^T over this wave's features; LDS reads run one row tile ahead
#pragma unroll
    for (int m = 0; m < NKH; ++m) sf[m] = acc_pair_frag<T>(S[2 * m], S[2 * m + 1]);
    f32x4 R[4];
    Frag<T> kf[2][NKH];
#pragma unroll
    for (int m = 0; m < NKH; ++m) kf[0][m] = ld_frag(Kb + c0 + 32 * m, LDQ);
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      if (J + 1 < 4)
#pragma unroll
        for (int m = 0; m < NKH; ++m) kf[(J + 1) & 1][m] = ld_frag(Kb + 16 * (J + 1) * LDQ + c0 + 32 * m, LDQ);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 acc = zero4();
#pragma unroll
      for (int m = 0; m < NKH; ++m) mma(acc, kf[J & 1][m], sf[m]);
      R[J] = acc;
    }
    if constexpr (NH > 1) {
      // sum the NH partial products of this value slice, in a fixed order so
      // every wave of the slice holds bit-identical P
#pragma unroll
      for (int J = 0; J < 4; ++J) sX[(w * 4 + J) * 64 + l] = R[J];
      lds_barrier();
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        f32x4 sum = sX[((pr * NH) * 4 + J) * 64 + l];
#pragma unroll
        for (int hh = 1; hh < NH; ++hh) sum += sX[((pr * NH + hh) * 4 + J) * 64 + l];
        R[J] = sum;
      }
    }
    // R = beta V - beta e^gamma P; V rows 32 m + 4 g4 + r and 32 m + 16 + 4 g4 + r
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const Frag<T> vf = ld_frag_tr_acc(sV[buf] + 32 * m * LDV + 16 * pr, LDV);
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int J = 2 * m + hh;
        const f32x4 bg = *reinterpret_cast<const f32x4*>(&sCf[buf][0][16 * J + 4 * g4]);
        const f32x4 bj = *reinterpret_cast<const f32x4*>(&sCf[buf][1][16 * J + 4 * g4]);
#pragma unroll
        for (int r = 0; r < 4; ++r) R[J][r] = bj[r] * frag_elem(vf, 4 * hh + r) - bg[r] * R[J][r];
      }
    }
    // U = Tm R (Tm rows are stored in acc_pos order)
    const Frag<T> rf0 = acc_pair_frag<T>(R[0], R[1]);
    const Frag<T> rf1 = acc_pair_frag<T>(R[2], R[3]);
    f32x4 U[4];
#pragma unroll
    for (int I = 0; I < 4; ++I) {
      U[I] = zero4();
      mma(U[I], ld_frag(sT[buf] + 16 * I * LDT, LDT), rf0);
      mma(U[I], ld_frag(sT[buf] + 16 * I * LDT + 32, LDT), rf1);
    }
    // U^T (kept for the write-back), then U e^{gamma_C - gamma_i}
    uf[0] = acc_pair_frag<T>(U[0], U[1]);
    uf[1] = acc_pair_frag<T>(U[2], U[3]);
#pragma unroll
    for (int I = 0; I < 4; ++I) U[I] *= *reinterpret_cast<const f32x4*>(&sCf[buf][2][16 * I + 4 * g4]);
    const Frag<T> ud0 = acc_pair_frag<T>(U[0], U[1]);
    const Frag<T> ud1 = acc_pair_frag<T>(U[2], U[3]);
    const float eC = sCf[buf][3][0];
    constexpr int TB = NCT < 4 ? NCT : 4;  // key-feature tiles per batch of transposing reads
    Frag<T> tf[2][TB][2];
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      tf[0][t][0] = ld_frag_tr_acc_pair(Kb + c0, LDQ, t);
      tf[0][t][1] = ld_frag_tr_acc_pair(Kb + 32 * LDQ + c0, LDQ, t);
    }
#pragma unroll
    for (int tb = 0; tb < NCT / TB; ++tb) {
      if (tb + 1 < NCT / TB)
#pragma unroll
        for (int t = 0; t < TB; ++t) {
          const int tc = TB * (tb + 1) + t;
          tf[(tb + 1) & 1][t][0] = ld_frag_tr_acc_pair(Kb + c0, LDQ, tc);
          tf[(tb + 1) & 1][t][1] = ld_frag_tr_acc_pair(Kb + 32 * LDQ + c0, LDQ, tc);
        }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < TB; ++t) {
        const int tc = TB * tb + t;
        S[tc] *= eC;
        mma(S[tc], tf[tb & 1][t][0], ud0);
        mma(S[tc], tf[tb & 1][t][1], ud1);
      }
    }
  };

  if (NL > 0) prefetch(st, 0);
  for (int ci = 0; ci < NL; ++ci) step(st, ci);

  if (NL > 0) write_back(NL - 1);
  if (a.ST) {
#pragma unroll
    for (int tc = 0; tc < NCT; ++tc)
      *reinterpret_cast<f32x4*>(a.ST + ((size_t)bh * a.dv + v) * DK + c0 + pair_feat(tc, g4)) = S[tc];
  }
}

// The same recurrence for bf16 with the chunk operands streamed straight into
// LDS (global_load_lds_dwordx4), NSTAGE - 1 chunks ahead, through a ring of
// NSTAGE stages: K (64 x DK), Tm (64 x 64), the V slice (64 x BVS) and the
// four coefficient rows.  No registers hold prefetched data and no
// instructions copy it; the vector-memory counter is waited on explicitly,
// with the chunk stores of the NSTAGE - 1 previous chunks allowed to remain in
// flight.  Rows are
// unpadded, so K and Tm are stored with their 16-byte pieces permuted per row
// (an XOR of the piece index) to keep the fragment reads free of bank
// conflicts: piece p of K row r sits at p ^ kswz(r), of Tm row r at p ^ tswz(r).
__device__ __forceinline__ int kswz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int tswz(int r) { return (r >> 1) & 7; }

template <int X>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(X) : "memory");
}
// s_waitcnt vmcnt(n) for a wave-uniform n in 0..47 (the counter field is an
// immediate: one scalar branch to the matching wait)
__device__ __forceinline__ void wait_vm_n(int n) {
  switch (n) {
#define CCQ_WAIT_CASE(i) \
  case i:                \
    wait_vm<i>();        \
    break;
#define CCQ_WAIT_CASE8(i) \
  CCQ_WAIT_CASE(i) CCQ_WAIT_CASE(i + 1) CCQ_WAIT_CASE(i + 2) CCQ_WAIT_CASE(i + 3) CCQ_WAIT_CASE(i + 4) \
  CCQ_WAIT_CASE(i + 5) CCQ_WAIT_CASE(i + 6) CCQ_WAIT_CASE(i + 7)
    CCQ_WAIT_CASE8(0) CCQ_WAIT_CASE8(8) CCQ_WAIT_CASE8(16) CCQ_WAIT_CASE8(24) CCQ_WAIT_CASE8(32) CCQ_WAIT_CASE8(40)
#undef CCQ_WAIT_CASE8
#undef CCQ_WAIT_CASE
    default:
      wait_vm<0>();
      break;
  }
}

// RS (reduce-scatter exchange): instead of every wave of a value tile reading
// all NH x 4 partial products and forming all of R, wave hq sums the partials
// of its own 4 / NH token tiles (the same fixed order), forms those tiles of R
// from its own rows of V and of the coefficients, and writes them as bf16 in
// the layout of the operand fragments of U = Tm R; after a second barrier every
// wave reads the two fragments.  R enters the product as bf16 either way.
// RSU (with RS): U = Tm R is split the same way: wave hq forms only the rows
// of its own token tiles, stores them as its part of U^T, and shares them,
// times e^{gamma_C - gamma}, as bf16 operand fragments for the state update.
template <int DK, int NPR, int NH, int NSTAGE, bool RS = false, bool RSU = false>
__global__ __launch_bounds__(64 * NPR * NH, 1) void gdn_state_dma_kernel(const GdnArgs a) {
  typedef bf16_t T;
  typedef __attribute__((address_space(3))) void lds_void;
  constexpr int C = kChunk, NW = NPR * NH, BVS = 16 * NPR;
  constexpr int DKH = DK / NH, NCT = DKH / 16, NKH = DKH / 32;
  constexpr int RB = DK * 2;                                  // K row bytes
  constexpr int KB = C * RB, TB = C * C * 2, VB = C * BVS * 2, FB = 4 * C * 4;
  constexpr int NIK = KB / 1024, NIT = TB / 1024, NIV = VB / 1024;
  constexpr int NIVW = (NIV + NW - 1) / NW;                   // V pieces per wave (some idle)
  constexpr int NIW = NIK / NW + NIT / NW + NIVW + 1;         // 1 KB pieces per wave and chunk
  constexpr int SB = KB + TB + VB + FB;
  constexpr int XB = NH > 1 ? NW * 4 * 64 * 16 : 16;
  constexpr int XR = (RS ? NPR * 2 * 64 * 16 : 0) * (RSU ? 2 : 1);  // bf16 R (RSU: and U) fragments
  constexpr int NSU = NH == 1 ? 2 : 1;                         // U^T stores per wave per chunk
  static_assert(DK == 128 || DK == 256, "key width");
  static_assert(NH == 1 || NH == 2 || NH == 4, "key split");
  static_assert(NSTAGE == 2 || NSTAGE == 3, "ring depth");
  static_assert(NKH >= 1 && VB % 1024 == 0, "tiles");
  static_assert(!RS || NH > 1, "the reduce-scatter exchange splits the keys");
  static_assert(!RSU || RS, "the split U builds on the split R");
  static_assert(NIV % NW == 0 || NW % NIV == 0, "V pieces over the waves");
  __shared__ __align__(1024) char smem[NSTAGE * SB + XB + XR];
  f32x4* const sX = reinterpret_cast<f32x4*>(smem + NSTAGE * SB);
  T* const sR = reinterpret_cast<T*>(smem + NSTAGE * SB + XB);
  T* const sU = sR + NPR * 2 * 64 * 8;  // RSU: fragments of U diag(e^{gamma_C - gamma})

  const int nvt = a.dv / BVS;
  const int N = (a.T + C - 1) / C;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  // heads in head-major order: the workgroups of consecutive logical blocks
  // (one compute-unit cluster) then hold one head of every sequence, which
  // balances the clusters when a packed batch's sequences differ in length
  const int hm = lb / nvt;
  const int bh = (hm % a.B) * a.H + hm / a.B;
  const int l = lane_id(), g4 = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pr = w / NH, hq = w % NH;
  const int v0 = (lb % nvt) * BVS;
  const int v = v0 + 16 * pr + c16;
  const int c0 = hq * DKH;
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  const int NL = (sq.len + C - 1) / C;  // chunks walked (a packed sequence's own)
  const T* k = static_cast<const T*>(a.k);
  const T* vin = static_cast<const T*>(a.v);
  const T* Tg = static_cast<const T*>(a.Tm);

  // chunk ci into stage ci % NSTAGE.  Piece i of each operand goes to wave
  // i % NW, so every wave issues the same number of pieces of each kind (a
  // piece that not every wave can have is shared out by lanes).  Addresses
  // are a per-chunk base (uniform) plus a 32-bit per-lane offset; rows past
  // the end of the sequence read row nrow - 1 (finite data; the chunk
  // transform zeroes their contribution).
  static_assert(NIK % NW == 0 && NIT % NW == 0 && 64 % NW == 0, "piece split");
  // the K pieces [it0, it1) of this wave
  auto issue_k = [&](int ci, int it0, int it1) {
    char* sb = smem + (ci % NSTAGE) * SB;
    const int r0 = ci * C, nrow = min(C, sq.len - r0);
    const int hs = a.H * DK;
    const T* kb = k + seq_off(sq, r0, h, a.H, DK);
#pragma unroll
    for (int it = 0; it < NIK / NW; ++it) {
      if (it < it0 || it >= it1) continue;
      constexpr int CPR = DK / 8;
      const int ins = it * NW + w, row = ins * (64 / CPR) + l / CPR;
      const int off = min(row, nrow - 1) * hs + 8 * ((l % CPR) ^ kswz(row));
      __builtin_amdgcn_global_load_lds((const void*)(kb + off), (lds_void*)(sb + ins * 1024), 16, 0, 0);
    }
  };
  // the Tm, V and coefficient pieces of this wave
  auto issue_rest = [&](int ci) {
    char* sb = smem + (ci % NSTAGE) * SB;
    const int r0 = ci * C, nrow = min(C, sq.len - r0);
    const int hv = a.H * a.dv;
    const T* tb = Tg + ((size_t)bh * N + ci) * C * C;
    const T* vb = vin + seq_off(sq, r0, h, a.H, a.dv) + v0;
#pragma unroll
    for (int it = 0; it < NIT / NW; ++it) {
      const int ins = it * NW + w, row = ins * 8 + l / 8;
      const int off = row * C + 8 * ((l % 8) ^ tswz(row));
      __builtin_amdgcn_global_load_lds((const void*)(tb + off), (lds_void*)(sb + KB + ins * 1024), 16, 0, 0);
    }
    {
      // with fewer V pieces than waves, NW / NIV waves share a piece, each
      // loading its own lanes of it (lane i of a piece lands at its base + 16 i
      // whichever lanes are active)
      constexpr int CPR = BVS / 8, SH = NIV >= NW ? 1 : NW / NIV, LPW = 64 / SH;
#pragma unroll
      for (int it = 0; it < NIVW; ++it) {
        const int ins = SH == 1 ? it * NW + w : w / SH, row = ins * (64 / CPR) + l / CPR;
        if (SH == 1 || l / LPW == w % SH) {
          const int off = min(row, nrow - 1) * hv + 8 * (l % CPR);
          __builtin_amdgcn_global_load_lds((const void*)(vb + off), (lds_void*)(sb + KB + TB + ins * 1024), 16, 0, 0);
        }
      }
    }
    // the coefficient rows, one piece shared the same way by all the waves
    if (l / (64 / NW) == w)
      __builtin_amdgcn_global_load_lds((const void*)(a.gam + (((size_t)bh * N + ci) * 5 + 1) * C + 4 * l),
                                       (lds_void*)(sb + KB + TB + VB), 16, 0, 0);
  };
  auto issue = [&](int ci) {
    issue_k(ci, 0, NIK / NW);
    issue_rest(ci);
  };
  // stores per wave of chunk c: S_r (every sstride-th chunk) and U^T
  auto nstore = [&](int c) { return (c % a.sstride == 0 ? NKH : 0) + NSU; };
  // wait until chunk ci has landed: the pieces and stores issued after its own
  // may stay in flight (three stages: stores of chunk ci - 2, pieces of
  // ci + 1, stores of ci - 1; two stages: stores of ci - 1)
  auto wait_chunk = [&](int ci) {
    int n = ci >= 1 ? nstore(ci - 1) : 0;
    if constexpr (NSTAGE == 3) n += (ci >= 2 ? nstore(ci - 2) : 0) + (ci + 1 < NL ? NIW : 0);
    wait_vm_n(n);
  };

#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < NL) issue(s);

  // S^T[c][v] in pair order: c = c0 + pair_feat(tc, g4) + r, so that the
  // packed operand of tiles 2m, 2m + 1 holds 8 consecutive features per lane
  // group (the states are stored so, and K is read with plain 16-byte reads)
  f32x4 S[NCT];
#pragma unroll
  for (int tc = 0; tc < NCT; ++tc) {
    if (a.S0)
      S[tc] = *reinterpret_cast<const f32x4*>(a.S0 + ((size_t)bh * a.dv + v) * DK + c0 + pair_feat(tc, g4));
    else
      S[tc] = zero4();
  }

  const int vt = (v0 >> 4) + pr;
  T* st_base = static_cast<T*>(a.states) + (((size_t)vt * (DK / 32) + hq * NKH) * 16 + c16) * 32 + 8 * g4;
  T* u_base = static_cast<T*>(a.U) + ((size_t)vt * 2 * 16 + c16) * 32 + 8 * g4;

  for (int ci = 0; ci < NL; ++ci) {
    const char* sb = smem + (ci % NSTAGE) * SB;
    const char* Kb = sb;
    const T* Tb = reinterpret_cast<const T*>(sb + KB);
    const T* Vb = reinterpret_cast<const T*>(sb + KB + TB);
    const float* Fb = reinterpret_cast<const float*>(sb + KB + TB + VB);
    wait_chunk(ci);
    lds_barrier();  // chunk ci visible; stage (ci - 1) % NSTAGE and the exchange area released
    // chunk ci + NSTAGE - 1 goes out in pieces between this chunk's first
    // products (their issue then overlaps the matrix cores' work), all of it
    // before this chunk's stores, so the counted waits stay as they are
    const bool ahead = ci + NSTAGE - 1 < NL;
    constexpr int KPJ = (NIK / NW + 3) / 4;  // K pieces after each token tile of P

    // P = K S_r^T over this wave's features: K rows 16 J + c16, features in
    // natural order (piece (c0 + 32 m) / 8 + g4, one 16-byte read)
    Frag<T> sf[NKH];
#pragma unroll
    for (int m = 0; m < NKH; ++m) sf[m] = acc_pair_frag<T>(S[2 * m], S[2 * m + 1]);
    const int ks = kswz(c16);
    auto kfrag = [&](int J, int m) {
      const char* row = Kb + (16 * J + c16) * RB;
      const int p0 = (c0 + 32 * m) / 8 + g4;
      Frag<T> f;
      f.v = *reinterpret_cast<const bf16x8*>(row + 16 * (p0 ^ ks));
      return f;
    };
    // the V slice, transposed (issued now, waited for where used); RS: the
    // rows of this wave's token tiles only (tile J is rows 16 J + 4 g4 + r)
    constexpr int JPW = RS ? 4 / NH : 4;
    const int J0 = RS ? hq * JPW : 0;
    Frag<T> vf[2];
    bf16x4 vw[RS ? JPW : 1];
    {
      const int j = c16;
      const char* pv = reinterpret_cast<const char*>(Vb) + (4 * g4 + (j >> 2)) * (2 * BVS) + 32 * pr + 8 * (j & 3);
      if constexpr (RS) {
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) vw[jj] = ds_read_tr16_asm(pv + 16 * (J0 + jj) * 2 * BVS);
      } else {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const bf16x4 lo = ds_read_tr16_asm(pv + 32 * m * 2 * BVS);
          const bf16x4 hi = ds_read_tr16_asm(pv + (32 * m + 16) * 2 * BVS);
          vf[m].v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
      }
    }
    f32x4 R[4];
    {
      Frag<T> kf[2][NKH];
#pragma unroll
      for (int m = 0; m < NKH; ++m) kf[0][m] = kfrag(0, m);
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        if (J + 1 < 4)
#pragma unroll
          for (int m = 0; m < NKH; ++m) kf[(J + 1) & 1][m] = kfrag(J + 1, m);
        __builtin_amdgcn_sched_barrier(0);
        f32x4 acc = zero4();
#pragma unroll
        for (int m = 0; m < NKH; ++m) mma(acc, kf[J & 1][m], sf[m]);
        R[J] = acc;
        if (ahead) issue_k(ci + NSTAGE - 1, J * KPJ, (J + 1) * KPJ);
      }
    }
    if (ahead) issue_rest(ci + NSTAGE - 1);
    // coefficients and Tm rows, read now so that their latency overlaps the
    // exchange
    constexpr int IPW = RSU ? JPW : 4;  // the token tiles of U this wave forms
    const int I0 = RSU ? J0 : 0;
    Frag<T> tfr[IPW][2];
    f32x4 bg[JPW], bj[JPW], dd[IPW];  // bg, bj: the token tiles this wave forms R for
#pragma unroll
    for (int jj = 0; jj < JPW; ++jj) {
      bg[jj] = *reinterpret_cast<const f32x4*>(Fb + 16 * (J0 + jj) + 4 * g4);
      bj[jj] = *reinterpret_cast<const f32x4*>(Fb + C + 16 * (J0 + jj) + 4 * g4);
    }
#pragma unroll
    for (int ii = 0; ii < IPW; ++ii) dd[ii] = *reinterpret_cast<const f32x4*>(Fb + 2 * C + 16 * (I0 + ii) + 4 * g4);
    const float eC = Fb[3 * C];
    {
      const int ts = tswz(c16);
#pragma unroll
      for (int ii = 0; ii < IPW; ++ii)
#pragma unroll
        for (int q = 0; q < 2; ++q)
          tfr[ii][q].v = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(Tb) +
                                                          (16 * (I0 + ii) + c16) * 128 + 16 * ((4 * q + g4) ^ ts));
    }
    Frag<T> rf0, rf1;  // R as the bf16 operand of U = Tm R (tiles 0, 1 and 2, 3)
    if constexpr (RS) {
      // this wave's token tiles: the NH partials summed in the fixed order,
      // R = beta V - beta e^gamma P, written as bf16 where fragment J / 2 of the
      // slice keeps tile J in its lane's elements 4 (J % 2) .. + 3
#pragma unroll
      for (int J = 0; J < 4; ++J) sX[(w * 4 + J) * 64 + l] = R[J];
      lds_barrier();  // (also completes this wave's V and coefficient reads)
#pragma unroll
      for (int jj = 0; jj < JPW; ++jj) asm volatile("" : "+v"(vw[jj]));
#pragma unroll
      for (int jj = 0; jj < JPW; ++jj) {
        const int J = J0 + jj;
        f32x4 sum = sX[((pr * NH) * 4 + J) * 64 + l];
#pragma unroll
        for (int hh = 1; hh < NH; ++hh) sum += sX[((pr * NH + hh) * 4 + J) * 64 + l];
        bf16x4 y;
#pragma unroll
        for (int r = 0; r < 4; ++r) y[r] = static_cast<bf16_t>(bj[jj][r] * f32(vw[jj][r]) - bg[jj][r] * sum[r]);
        *reinterpret_cast<bf16x4*>(sR + ((pr * 2 + (J >> 1)) * 64 + l) * 8 + 4 * (J & 1)) = y;
      }
      lds_barrier();
      rf0.v = *reinterpret_cast<const bf16x8*>(sR + ((pr * 2) * 64 + l) * 8);
      rf1.v = *reinterpret_cast<const bf16x8*>(sR + ((pr * 2 + 1) * 64 + l) * 8);
    } else if constexpr (NH > 1) {
      // sum the NH partial products of this value slice, in a fixed order so
      // every wave of the slice holds bit-identical P
#pragma unroll
      for (int J = 0; J < 4; ++J) sX[(w * 4 + J) * 64 + l] = R[J];
      lds_barrier();
      f32x4 part[NH][4];
#pragma unroll
      for (int hh = 0; hh < NH; ++hh)
#pragma unroll
        for (int J = 0; J < 4; ++J) part[hh][J] = sX[((pr * NH + hh) * 4 + J) * 64 + l];
#pragma unroll
      for (int J = 0; J < 4; ++J) {
        f32x4 sum = part[0][J];
#pragma unroll
        for (int hh = 1; hh < NH; ++hh) sum += part[hh][J];
        R[J] = sum;
      }
    }
    // K^T of this wave's features for the update, in the pair order of the
    // state tiles (rows 4 g4 + j / 4 (+ 16) of each 32-token half, features
    // c0 + pair_feat(t, j % 4): piece (c0 + 32 (t / 2)) / 8 + j % 4, half t % 2),
    // issued now so that they arrive while R and U are formed
    Frag<T> tf[NCT][2];
    {
      const int j = c16, rr = 4 * g4 + (j >> 2), rs = kswz(rr);
#pragma unroll
      for (int t = 0; t < NCT; ++t)
#pragma unroll
        for (int kq = 0; kq < 2; ++kq) {
          const int p = (c0 + 32 * (t >> 1)) / 8 + (j & 3), hb = (t & 1) * 8;
          const char* pl = Kb + (32 * kq + rr) * RB + 16 * (p ^ rs) + hb;
          const bf16x4 lo = ds_read_tr16_asm(pl);
          const bf16x4 hi = ds_read_tr16_asm(pl + 16 * RB);
          tf[t][kq].v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
    }
    if constexpr (!RS) {
      lds_wait_but<(4 * NCT < 15 ? 4 * NCT : 15)>(vf);  // at most 15 LDS reads stay in flight
      // R = beta V - beta e^gamma P
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int J = 2 * m + hh;
#pragma unroll
          for (int r = 0; r < 4; ++r) R[J][r] = bj[J][r] * frag_elem(vf[m], 4 * hh + r) - bg[J][r] * R[J][r];
        }
      rf0 = acc_pair_frag<T>(R[0], R[1]);
      rf1 = acc_pair_frag<T>(R[2], R[3]);
    }
    // U = Tm R (Tm rows are stored in acc_pos order)
    f32x4 U[IPW];
#pragma unroll
    for (int ii = 0; ii < IPW; ++ii) {
      U[ii] = zero4();
      mma(U[ii], tfr[ii][0], rf0);
      mma(U[ii], tfr[ii][1], rf1);
    }
    Frag<T> uf[2], ud0, ud1;
    bf16x4 uw[IPW];  // RSU: this wave's tiles of U as bf16, its part of U^T
    if constexpr (RSU) {
      // tile I lives in elements 4 (I % 2) .. + 3 of fragment I / 2
#pragma unroll
      for (int ii = 0; ii < IPW; ++ii) {
        const int I = I0 + ii;
        bf16x4 y;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          uw[ii][r] = static_cast<bf16_t>(U[ii][r]);
          y[r] = static_cast<bf16_t>(U[ii][r] * dd[ii][r]);
        }
        *reinterpret_cast<bf16x4*>(sU + ((pr * 2 + (I >> 1)) * 64 + l) * 8 + 4 * (I & 1)) = y;
      }
      lds_barrier();
      ud0.v = *reinterpret_cast<const bf16x8*>(sU + ((pr * 2) * 64 + l) * 8);
      ud1.v = *reinterpret_cast<const bf16x8*>(sU + ((pr * 2 + 1) * 64 + l) * 8);
    } else {
      uf[0] = acc_pair_frag<T>(U[0], U[1]);
      uf[1] = acc_pair_frag<T>(U[2], U[3]);
#pragma unroll
      for (int I = 0; I < 4; ++I) U[I] *= dd[I];
      ud0 = acc_pair_frag<T>(U[0], U[1]);
      ud1 = acc_pair_frag<T>(U[2], U[3]);
    }
    // S^T <- e^{gamma_C} S^T + K^T diag(e^{gamma_C - gamma}) U
#pragma unroll
    for (int t = 1; t < NCT; ++t) lds_wait(tf[t]);
#pragma unroll
    for (int tc = 0; tc < NCT; ++tc) {
      S[tc] *= eC;
      mma(S[tc], tf[tc][0], ud0);
      mma(S[tc], tf[tc][1], ud1);
    }
    // S_r and U^T of this chunk, fragment-native (1 KB per value tile and k step)
    {
      T* st_out = st_base + ((size_t)bh * N + ci) * a.dv * DK;
      if (ci % a.sstride == 0)
#pragma unroll
        for (int m = 0; m < NKH; ++m) store_frag(st_out + 16 * 32 * m, sf[m]);
      T* u_out = u_base + ((size_t)bh * N + ci) * a.dv * C;
      if constexpr (RSU && IPW == 2) {
        // two waves: fragment hq whole
        *reinterpret_cast<bf16x8*>(u_out + 16 * 32 * hq) =
            bf16x8{uw[0][0], uw[0][1], uw[0][2], uw[0][3], uw[1][0], uw[1][1], uw[1][2], uw[1][3]};
      } else if constexpr (RSU) {
        *reinterpret_cast<bf16x4*>(u_out + 16 * 32 * (I0 >> 1) + 4 * (I0 & 1)) = uw[0];
      } else if constexpr (NH == 1) {
        store_frag(u_out, uf[0]);
        store_frag(u_out + 16 * 32, uf[1]);
      } else if constexpr (NH == 2) {
        store_frag(u_out + 16 * 32 * hq, hq == 0 ? uf[0] : uf[1]);
      } else {
        // four waves: one 8-byte half of one fragment each
        const bf16x8 x = (hq >> 1) == 0 ? uf[0].v : uf[1].v;
        const bf16x4 y = (hq & 1) == 0 ? bf16x4{x[0], x[1], x[2], x[3]} : bf16x4{x[4], x[5], x[6], x[7]};
        *reinterpret_cast<bf16x4*>(u_out + 16 * 32 * (hq >> 1) + 4 * (hq & 1)) = y;
      }
    }
  }

  if (a.ST) {
    wait_vm<0>();
#pragma unroll
    for (int tc = 0; tc < NCT; ++tc)
      *reinterpret_cast<f32x4*>(a.ST + ((size_t)bh * a.dv + v) * DK + c0 + pair_feat(tc, g4)) = S[tc];
  }
}

// Outputs of a group of consecutive chunks (eight waves).  Per chunk the
// decayed, masked scores
//   P_ij = e^{gamma_i - gamma_j} (q_i . k_j)  (j <= i)
// are formed once (ten nonzero 16 x 16 tiles over the waves) and kept in LDS;
// wave w then owns VPW value tiles for IPW token tiles and forms, transposed,
//   O^T = e^{gamma_i} (S_r Q^T) + U^T P^T,
// with rows of U^T read straight from global memory as MFMA operands.  S_r
// of the group's first chunk is read the same way; for the later chunks each
// wave carries its rows of S forward itself,
//   S_{r+1} = e^{gamma_C} S_r + U^T diag(e^{gamma_C - gamma}) K,
// so the state pass stores one state per group.  S is held as bf16 operand
// fragments in natural feature order; a fragment's 8 elements are exactly
// the lane's entries of two pair-ordered accumulator tiles (tiles 2m, 2m + 1
// of ld_frag_tr_acc_pair), so the update unpacks, accumulates and repacks in
// place.
template <typename T, int DK, int VPW, int IPW, bool CARRY>
__global__ __launch_bounds__(kOutThreads, 1) void gdn_out_kernel(const GdnOutArgs a) {
  constexpr int C = kChunk;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDP = C + P;
  constexpr int NK = DK / 32;
  constexpr int NIG = 4 / IPW;  // token-tile groups
  constexpr int NVG = 8 / NIG;  // value-tile groups
  static_assert(NVG * NIG == 8, "wave split");

  __shared__ __align__(16) T sQ[C * LDQ];
  __shared__ __align__(16) T sK[C * LDQ];
  __shared__ __align__(16) T sP[C * LDP];  // P[i][acc_pos(j)]
  __shared__ __align__(16) float sGam[C];
  __shared__ __align__(16) float sDd[C + 4];  // e^{gamma_C - gamma_j}; e^{gamma_C} at C
  __shared__ float sRk[C];                    // raw keys: row scales of the scores

  const int N = (a.T + C - 1) / C;
  const int R = CARRY ? a.group : 1, NGR = (N + R - 1) / R;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int hm = lb / NGR, cb = (lb % NGR) * R;
  const int bh = (hm % a.B) * a.H + hm / a.B;  // head-major, as the state pass
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  const int ce = min((sq.len + C - 1) / C, cb + R);  // a packed sequence's own chunks
  if (cb >= ce) return;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const int vg = w % NVG, ig = NIG == 1 ? 0 : w / NVG;  // (uniform: no lane-masked branch on the tile)
  const size_t gstride = (size_t)a.H * DK;
  T* o = static_cast<T*>(a.o);

  Frag<T> sfr[VPW][NK];
  for (int ci = cb; ci < ce; ++ci) {
    const int r0 = ci * C;
    const int nrow = (sq.len - r0) < C ? (sq.len - r0) : C;
    const bool carry = CARRY && ci + 1 < ce;
    {
      RowTile<T, DK, kOutThreads> rq, rk;
      rq.load(static_cast<const T*>(a.qc) + seq_off(Seq{(long long)b * a.T, sq.len}, r0, h, a.H, DK), gstride,
              nrow);  // q_clean: the workspace's padded rows
      rk.load(static_cast<const T*>(a.k) + seq_off(sq, r0, h, a.H, DK), gstride, nrow);
      const float* gm = a.gam + ((size_t)bh * N + ci) * 5 * C;
      if (tid < C) sGam[tid] = gm[tid];
      if (a.rk && tid < C) sRk[tid] = a.rk[seq_idx(sq, r0 + (tid < nrow ? tid : nrow - 1), h, a.H)];
      if (carry && tid < C + 1) sDd[tid] = tid < C ? gm[3 * C + tid] : gm[4 * C];
      rq.store(sQ, LDQ);
      rk.store(sK, LDQ);
    }
    // (the barriers order LDS only: a __syncthreads() fence would also wait
    // for the output stores in flight)
    lds_barrier();

    // this wave's S_r (first chunk of the group) and U^T fragments
    // (fragment-native, 1 KB each), issued after the staging of q and k so
    // that they arrive while the score tiles are formed
    if (ci == cb) {
      const T* Sg = static_cast<const T*>(a.states) + ((size_t)bh * N + ci) * a.dv * DK;
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
        for (int m = 0; m < NK; ++m)
          sfr[vt][m] = ld_frag_global(Sg + ((size_t)(vg * VPW + vt) * NK + m) * 16 * 32, 32);
    }
    const T* Ug = static_cast<const T*>(a.U) + ((size_t)bh * N + ci) * a.dv * C;
    Frag<T> ufr[VPW][2];
#pragma unroll
    for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
      for (int m = 0; m < 2; ++m) ufr[vt][m] = ld_frag_global(Ug + ((size_t)(vg * VPW + vt) * 2 + m) * 16 * 32, 32);

    // P tiles: ten lower tiles (I >= J) over the waves, the six upper ones zero;
    // computed transposed (row j, column i) and stored as rows i
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
          x[r] = j <= i ? sc[r] * __expf(gi - sGam[j]) * (a.rk ? sRk[j] : 1.f) : 0.f;
        }
      }
      store4(sP + i * LDP + acc_pos(16 * J + 4 * g4), x[0], x[1], x[2], x[3]);
    }
    lds_barrier();

#pragma unroll
    for (int it = 0; it < IPW; ++it) {
      const int I = ig * IPW + it;
      const int i = 16 * I + c16;
      // S_r Q^T one k step at a time (one q fragment live), all value tiles
      f32x4 acc[VPW];
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) acc[vt] = zero4();
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        const Frag<T> qf = ld_frag(sQ + 16 * I * LDQ + 32 * m, LDQ);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) mma(acc[vt], sfr[vt][m], qf);
      }
      const Frag<T> pf0 = ld_frag(sP + 16 * I * LDP, LDP);
      const Frag<T> pf1 = ld_frag(sP + 16 * I * LDP + 32, LDP);
      const float ei = __expf(sGam[i]);
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) {
        acc[vt] *= ei;
        mma(acc[vt], ufr[vt][0], pf0);
        if (I >= 2) mma(acc[vt], ufr[vt][1], pf1);  // keys 32..63 precede row i only for I >= 2
        if (i < nrow) {
          const int vcol = 16 * (vg * VPW + vt) + 4 * g4;
          store4(o + seq_off(sq, r0 + i, h, a.H, a.dv) + vcol, a.scale * acc[vt][0], a.scale * acc[vt][1],
                 a.scale * acc[vt][2], a.scale * acc[vt][3]);
        }
      }
    }

    if constexpr (CARRY) if (carry) {
      // S_{r+1}^T = e^{gamma_C} S_r^T + K^T (diag(e^{gamma_C - gamma}) U): the
      // U^T fragments scaled per token (k slot 8 g4 + e is token 32 m + 4 g4 + e,
      // or + 16 for e >= 4), then per 32-feature block m the two pair-ordered
      // tiles of every value tile
      const float eC = sDd[C];
      Frag<T> ud[VPW][2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(sDd + 32 * m + 4 * g4);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(sDd + 32 * m + 16 + 4 * g4);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) {
          f32x4 x, y;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] = frag_elem(ufr[vt][m], r) * d0[r];
            y[r] = frag_elem(ufr[vt][m], 4 + r) * d1[r];
          }
          ud[vt][m] = acc_pair_frag<T>(x, y);
        }
      }
      // K^T fragments of block m + 1 are read while block m is updated (the
      // scheduling barrier keeps later blocks' reads from being hoisted)
      Frag<T> tf[2][2][2];
      auto load_tf = [&](Frag<T>(&f)[2][2], int m) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int kq = 0; kq < 2; ++kq) f[hh][kq] = ld_frag_tr_acc_pair(sK + 32 * kq * LDQ, LDQ, 2 * m + hh);
      };
      load_tf(tf[0], 0);
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        if (m + 1 < NK) load_tf(tf[(m + 1) & 1], m + 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) {
          f32x4 x, y;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] = eC * frag_elem(sfr[vt][m], r);
            y[r] = eC * frag_elem(sfr[vt][m], 4 + r);
          }
          mma(x, tf[m & 1][0][0], ud[vt][0]);
          mma(x, tf[m & 1][0][1], ud[vt][1]);
          mma(y, tf[m & 1][1][0], ud[vt][0]);
          mma(y, tf[m & 1][1][1], ud[vt][1]);
          sfr[vt][m] = acc_pair_frag<T>(x, y);
        }
      }
    }
    lds_barrier();  // q, k, P and the coefficients of this chunk released
  }
}

namespace {
template <typename T, int DK>
hipError_t run_tri(const TriArgs& a, hipStream_t st) {
  const int N = (a.T + kChunk - 1) / kChunk;
  const int nblk = a.B * a.H * N;
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_tri_kernel<T, DK>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK, int NPR, int NH>
hipError_t run_gdn_state_v(const GdnArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / (16 * NPR));
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_state_kernel<T, DK, NPR, NH>), dim3(nblk), dim3(64 * NPR * NH), 0, st, a);
  return hipGetLastError();
}
// Split the key features over as many waves (1, 2, 4 or 8, at least 32
// features each) as it takes to give every SIMD of the chip a wave, with four
// waves per workgroup where the split allows.
// LDS of the streamed kernel with a ring of `ns` stages
constexpr size_t gdn_dma_lds(int dk, int npr, int nh, int ns, bool rs, bool rsu) {
  return (size_t)ns * (kChunk * dk * 2 + kChunk * kChunk * 2 + kChunk * 16 * npr * 2 + 4 * kChunk * 4) +
         (nh > 1 ? (size_t)npr * nh * 4 * 64 * 16 : 16) + (rs ? (size_t)npr * 2 * 64 * 16 * (rsu ? 2 : 1) : 0);
}
// With a key split the exchange is the reduce-scatter form: bit-identical, and
// measured on the 1.3B shape 380 -> 362 us per forward call at T = 4096 and
// 915 -> 865 us at T = 20480.
template <int DK, int NPR, int NH, bool RS = (NH > 1), bool RSU = (NH > 1)>
hipError_t run_gdn_state_dma(const GdnArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dv / (16 * NPR));
  if (nblk == 0) return hipSuccess;
  // three stages where they fit in the compute unit's 160 KB of LDS
  constexpr int NS = gdn_dma_lds(DK, NPR, NH, 3, RS, RSU) <= 160 * 1024 ? 3 : 2;
  hipLaunchKernelGGL((gdn_state_dma_kernel<DK, NPR, NH, NS, RS, RSU>), dim3(nblk), dim3(64 * NPR * NH), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_gdn_state(const GdnArgs& a, hipStream_t st) {
  const long long slices = (long long)a.B * a.H * (a.dv / 16);
  constexpr int kSimds = 1024;
  if constexpr (sizeof(T) == 2 && (DK == 128 || DK == 256)) {
    // one workgroup per compute unit: at dk = 128, 64-wide value slices once
    // there are enough of them, so that the chip takes every slice in one
    // round (at dk = 256 that split would not fit the registers)
    if constexpr (DK == 128)
      if (slices >= kSimds && a.dv % 64 == 0) return run_gdn_state_dma<DK, 4, 2>(a, st);
    if (slices * 2 >= kSimds && a.dv % 32 == 0) return run_gdn_state_dma<DK, 2, 4>(a, st);
    // at most one value tile per compute unit at dk = 256 (long sequences of
    // few heads): one tile per workgroup over four waves, which beats eight
    // waves of the register-prefetch form (fewer partial products to exchange)
    if constexpr (DK == 256)
      if (slices <= kSimds / 4) return run_gdn_state_dma<DK, 1, 4>(a, st);
  }
  if (slices >= kSimds || DK < 64) return run_gdn_state_v<T, DK, 4, 1>(a, st);
  if (slices * 2 >= kSimds || DK < 128) return run_gdn_state_v<T, DK, 2, 2>(a, st);
  if constexpr (DK >= 128) {
    if (slices * 4 >= kSimds || DK < 256) return run_gdn_state_v<T, DK, 1, 4>(a, st);
  }
  if constexpr (DK >= 256) return run_gdn_state_v<T, DK, 1, 8>(a, st);
  return hipErrorInvalidValue;
}
template <typename T, int DK, int VPW, int IPW>
hipError_t run_gdn_out_v(const GdnOutArgs& a, hipStream_t st) {
  if (a.group < 1) return hipErrorInvalidValue;
  constexpr bool kCarry = DK * VPW * (int)sizeof(T) <= 1024;  // as gdn_out_carries
  if (!kCarry && a.group != 1) return hipErrorInvalidValue;
  const int N = (a.T + kChunk - 1) / kChunk;
  const int nblk = a.B * a.H * ((N + a.group - 1) / a.group);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gdn_out_kernel<T, DK, VPW, IPW, kCarry>), dim3(nblk), dim3(kOutThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_gdn_out(const GdnOutArgs& a, hipStream_t st) {
  switch (a.dv) {
    case 64: return run_gdn_out_v<T, DK, 1, 2>(a, st);
    case 128: return run_gdn_out_v<T, DK, 1, 4>(a, st);
    case 256: return run_gdn_out_v<T, DK, 2, 4>(a, st);
    case 512: return run_gdn_out_v<T, DK, 4, 4>(a, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

int gdn_out_group(int B, int H, int T, int dk, int dv, bool is_bf16) {
  // One workgroup (a compute unit's worth) walks its group's chunks in order
  // after reading one stored state, so the kernel takes about (rounds of 256
  // workgroups) x (group + 1) chunk steps: the group of 8, 4, 2 or 1 chunks
  // that minimises that, the largest on a tie (fewer stored states).  No
  // groups where a wave's share of S would not fit its registers beside the
  // output's.
  if (!gdn_out_carries(dk, dv, is_bf16)) return 1;
  const long long bh = (long long)B * H;
  const long long N = (T + kChunk - 1) / kChunk;
  int best = 1;
  long long best_cost = -1;
  for (int g = 1; g <= 8; g *= 2) {
    const long long rounds = (bh * ((N + g - 1) / g) + 255) / 256;
    const long long cost = rounds * (g + 1);
    if (best_cost < 0 || cost <= best_cost) {
      best_cost = cost;
      best = g;
    }
  }
  return best;
}

bool gdn_out_carries(int dk, int dv, bool is_bf16) {
  // a wave holds S for its value tiles (dv / 128 of them, at least one) and
  // all dk features as operand fragments: up to 64 registers
  const int vpw = dv / 128;
  return dk * (vpw < 1 ? 1 : vpw) * (is_bf16 ? 2 : 4) <= 1024;
}

bool gdn_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  if (is_bf16) return dv_ok && (dk == 64 || dk == 128 || dk == 256);
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gdn_tri(const TriArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_tri<bf16_t, 64>(a, st);
      case 128: return run_tri<bf16_t, 128>(a, st);
      case 256: return run_tri<bf16_t, 256>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_tri<float, 64>(a, st);
      case 128: return run_tri<float, 128>(a, st);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gdn_state(const GdnArgs& a, bool is_bf16, hipStream_t st) {
  if (is_bf16) {
    switch (a.dk) {
      case 64: return run_gdn_state<bf16_t, 64>(a, st);
      case 128: return run_gdn_state<bf16_t, 128>(a, st);
      case 256: return run_gdn_state<bf16_t, 256>(a, st);
    }
  } else {
    switch (a.dk) {
      case 64: return run_gdn_state<float, 64>(a, st);
      case 128: return run_gdn_state<float, 128>(a, st);
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
