// ccq_gla.hip -- GLA backbone chunk forward reading the cleaned queries.
//
// GLA (the cited backbone): S_t = S_{t-1} diag(e^{g_t}) + v_t k_t^T, o_t = S_t q_t.
// Within a chunk with inclusive log-decay prefix b_i = sum_{s<=i} g_s (per key
// channel) and entering state S_r:
//
//   o_i     = S_r (q_i * e^{b_i}) + sum_{j<=i} [sum_c q_i[c] k_j[c] e^{b_i[c]-b_j[c]}] v_j
//   S_{r+1} = S_r diag(e^{b_C}) + sum_j v_j (k_j * e^{b_C - b_j})^T
//
// gla_state_kernel carries a 64-channel tile of S through the chunks of a
// head (rows and columns of S evolve independently under the GLA write) and
// stores S_r for every chunk (a forward pass: for the first chunk of every
// output group); gla_out_kernel forms the outputs of every chunk, or of every
// group of chunks, in parallel.  The output uses a mid-chunk reference m = C/2: Qt = q * e^{b - b_m},
// Kt = k * e^{b_m - b}, so Qt Kt^T carries e^{b_i - b_j} with factors of at most
// e^{|b_m - b_i|} (a 32-token log-decay), and the inter-chunk read is
// Qt (S_r diag(e^{b_m}))^T.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

// State recurrence over the chunks of one head for 64 key channels and VB
// values.  Wave w owns channels c0 + 16 w .. + 15 (rows of S^T in its MFMA
// accumulators) for all VB values.  Per chunk the keys, gates and values are
// staged once (double-buffered LDS, one barrier); each wave then reads its
// channels' gates and keys transposed (lane = channel, 8 tokens per lane and
// k step), scans the gates in registers (8-token runs, then shuffles across
// the four lane groups) and forms the decayed keys k e^{b_C - b} directly as
// the MFMA operand of  S^T <- diag(e^{b_C}) S^T + Kd^T V.  S_r is written
// back one iteration late (all vector memory operations share one in-order
// counter, so a store just before the next loads are waited for would add
// its latency to every chunk).
//
// With kRev the same pass runs backwards for the training step: over the
// chunks from last to first it carries the state adjoint D = dL/dS_{r+1} and
// stores it for every chunk, with  D^T <- diag(e^{b_C}) D^T + s (Q e^{b})^T dO
// (a.k = q_clean, a.v = dO, a.states = the adjoints, a.scale = s).
template <typename T, typename TG, int NVT, bool kRev = false>
__global__ __launch_bounds__(kThreads, 1) void gla_state_kernel(const GlaStateArgs a) {
  constexpr int C = kChunk, BK = 64, VB = 16 * NVT;
  constexpr int P = Pad<T>::value, PG = Pad<TG>::value;
  constexpr int LDK = BK + P, LDG = BK + PG, LDV = VB + P;

  __shared__ __align__(16) T sK[2][C * LDK];
  __shared__ __align__(16) TG sG[2][C * LDG];
  __shared__ __align__(16) T sV[2][C * LDV];

  const int nkt = a.dk / BK, nvt = a.dv / VB;
  const int N = (a.T + C - 1) / C;
  const int SL = a.seg > 0 ? a.seg : N, NS = (N + SL - 1) / SL;  // segment length and count
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int vt = lb % nvt, kt = (lb / nvt) % nkt, sg = (lb / (nvt * nkt)) % NS, bh = lb / (nvt * nkt * NS);
  const int c0 = kt * BK, v0 = vt * VB;
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  // this segment's chunks (none past a packed sequence's end: the segment then
  // passes its entry state through unchanged, zero sum and unit decay)
  const int cb = sg * SL, ce = min((sq.len + C - 1) / C, cb + SL);
  const int w = wave_id(), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const T* k = static_cast<const T*>(a.k);
  const T* v = static_cast<const T*>(a.v);
  const TG* gate = static_cast<const TG*>(a.g);

  // S^T tiles: S[tv][r] = S[v][c], c = c0 + 16 w + 4 g4 + r, v = v0 + 16 tv + c16
  f32x4 S[NVT];
#pragma unroll
  for (int tv = 0; tv < NVT; ++tv) {
    const int vv = v0 + 16 * tv + c16;
    S[tv] = (a.S0 && sg == 0)
                ? *reinterpret_cast<const f32x4*>(a.S0 + ((size_t)bh * a.dv + vv) * a.dk + c0 + 16 * w + 4 * g4)
                : zero4();
  }

  // a chunk's keys, gates and values, prefetched into registers two chunks
  // ahead (two sets, alternating)
  struct Stage {
    RowTile<T, BK, kThreads, true> rk;
    RowScales<RowTile<T, BK, kThreads, true>> fk;  // raw keys: row scales (l2 normalisation)
    RowTile<TG, BK, kThreads, true> rg;
    RowTile<T, VB, kThreads, true> rv;
  };
  Stage sa, sb;
  auto prefetch = [&](Stage& st, int ci) {
    const int r0 = ci * C;
    const int nrow = (sq.len - r0) < C ? (sq.len - r0) : C;
    st.rk.load(k + seq_off(sq, r0, h, a.H, a.dk) + c0, (size_t)a.H * a.dk, nrow);
    if (a.rk) st.fk.load(a.rk + seq_idx(sq, r0, h, a.H), (size_t)a.H, nrow);
    st.rg.load(gate + seq_off(sq, r0, h, a.H, a.dk) + c0, (size_t)a.H * a.dk, nrow);
    st.rv.load(v + seq_off(sq, r0, h, a.H, a.dv) + v0, (size_t)a.H * a.dv, nrow);
  };
  f32x4 Sr[NVT];  // S_r kept for the deferred write-back
  // only the first chunk of each output group (a.group chunks) is read back
  const int grp = (!kRev && a.group > 1) ? a.group : 1;
  auto write_back = [&](int cw) {
    if (cw % grp != 0) return;
    T* st = static_cast<T*>(a.states) + (((size_t)bh * N + cw) * a.dv + v0) * a.dk + c0 + 16 * w + 4 * g4;
#pragma unroll
    for (int tv = 0; tv < NVT; ++tv)
      store4(st + (size_t)(16 * tv + c16) * a.dk, Sr[tv][0], Sr[tv][1], Sr[tv][2], Sr[tv][3]);
  };
  const int nch = ce - cb;
  auto chunk = [&](int it) { return kRev ? ce - 1 - it : cb + it; };
  if (nch > 0) prefetch(sa, chunk(0));
  if (nch > 1) prefetch(sb, chunk(1));
  float le = 0.f;  // log decay of this lane's channel since the segment began

  auto step = [&](Stage& st, int it) {
    const int ci = chunk(it);
    const int buf = it & 1;  // the other buffer was released at the previous barrier
    if (a.rk) st.fk.apply(st.rk);
    st.rk.store(sK[buf], LDK);
    st.rg.store(sG[buf], LDG);
    st.rv.store(sV[buf], LDV);
    if (it > 0) write_back(kRev ? ci + 1 : ci - 1);
    if (it + 2 < nch) prefetch(st, chunk(it + 2));
#pragma unroll
    for (int tv = 0; tv < NVT; ++tv) Sr[tv] = S[tv];
    // orders LDS only: a __syncthreads() fence would wait for the prefetch
    // just issued and for the state stores
    lds_barrier();

    // gates and keys of this wave's channels: lane = channel c0 + 16 w + c16,
    // tokens 32 m + 8 g4 + e
    const Frag<TG> gf0 = ld_frag_tr(sG[buf] + 16 * w, LDG);
    const Frag<TG> gf1 = ld_frag_tr(sG[buf] + 32 * LDG + 16 * w, LDG);
    const Frag<T> kf0 = ld_frag_tr(sK[buf] + 16 * w, LDK);
    const Frag<T> kf1 = ld_frag_tr(sK[buf] + 32 * LDK + 16 * w, LDK);
    float pb[2][8], tot[2], ex[2], half[2];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pb[0][e] = frag_elem(gf0, e) + (e ? pb[0][e - 1] : 0.f);
      pb[1][e] = frag_elem(gf1, e) + (e ? pb[1][e - 1] : 0.f);
    }
#pragma unroll
    for (int m = 0; m < 2; ++m) {  // scan of the 8-token totals over the four lane groups
      tot[m] = pb[m][7];
      float sc = tot[m];
      const float u1 = __shfl_up(sc, 16);
      if (g4 >= 1) sc += u1;
      const float u2 = __shfl_up(sc, 32);
      if (g4 >= 2) sc += u2;
      ex[m] = sc - tot[m];
      half[m] = __shfl(sc, 48 + c16);
    }
    const float bC = half[0] + half[1];
    if (a.cdec && vt == 0 && g4 == 0) a.cdec[((size_t)bh * N + ci) * a.dk + c0 + 16 * w + c16] = __expf(le);
    le += bC;
    Frag<T> kd0, kd1;  // forward: k e^{b_C - b}; reverse: s q e^{b}
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float b0 = ex[0] + pb[0][e], b1 = half[0] + ex[1] + pb[1][e];
      if constexpr (kRev) {
        set_frag_elem(kd0, e, a.scale * frag_elem(kf0, e) * __expf(b0));
        set_frag_elem(kd1, e, a.scale * frag_elem(kf1, e) * __expf(b1));
      } else {
        set_frag_elem(kd0, e, frag_elem(kf0, e) * __expf(bC - b0));
        set_frag_elem(kd1, e, frag_elem(kf1, e) * __expf(bC - b1));
      }
    }
    // S^T <- diag(e^{b_C}) S^T + Kd^T V; row c = 4 g4 + r of the tile needs e^{b_C[c]}
    f32x4 dec;
#pragma unroll
    for (int r = 0; r < 4; ++r) dec[r] = __expf(__shfl(bC, 4 * g4 + r));
#pragma unroll
    for (int tv = 0; tv < NVT; ++tv) {
      S[tv] *= dec;
      mma(S[tv], kd0, ld_frag_tr(sV[buf] + 16 * tv, LDV));
      mma(S[tv], kd1, ld_frag_tr(sV[buf] + 32 * LDV + 16 * tv, LDV));
    }
  };
  for (int it = 0; it < nch; it += 2) {
    step(sa, it);
    if (it + 1 < nch) step(sb, it + 1);
  }

  if (nch > 0) write_back(kRev ? cb : ce - 1);
  // the segment's total: the local state at its end and its decay (or, with
  // one segment, the final state)
  float* out = a.segsum ? a.segsum + ((size_t)bh * NS + sg) * a.dv * a.dk
                        : (a.ST ? a.ST + (size_t)bh * a.dv * a.dk : nullptr);  // one segment: sg = 0
  if (out) {
#pragma unroll
    for (int tv = 0; tv < NVT; ++tv) {
      const int vv = v0 + 16 * tv + c16;
      *reinterpret_cast<f32x4*>(out + (size_t)vv * a.dk + c0 + 16 * w + 4 * g4) = S[tv];
    }
  }
  if (a.segdec && vt == 0 && g4 == 0) a.segdec[((size_t)bh * NS + sg) * a.dk + c0 + 16 * w + c16] = __expf(le);
}

// Entry state of every segment of the GLA state pass, four elements per
// thread: E_0 = 0, E_{j+1} = E_j diag(segdec_j) + segsum_j, S_T = E_NS.
template <typename T>
__global__ __launch_bounds__(256) void gla_scan_kernel(const GlaScanArgs a) {
  const size_t DD = (size_t)a.dv * a.dk;
  const size_t e4 = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (e4 >= (size_t)a.B * a.H * DD) return;
  const size_t bh = e4 / DD, el = e4 % DD;
  const int c = (int)(el % a.dk);
  f32x4 x = zero4();
  for (int j = 0; j < a.NS; ++j) {
    const size_t so = bh * a.NS + j;
    if (j > 0) store4(static_cast<T*>(a.entries) + so * DD + el, x[0], x[1], x[2], x[3]);
    const f32x4 d = *reinterpret_cast<const f32x4*>(a.segdec + so * a.dk + c);
    const f32x4 s = *reinterpret_cast<const f32x4*>(a.segsum + so * DD + el);
    x = x * d + s;
  }
  if (a.ST) *reinterpret_cast<f32x4*>(a.ST + bh * DD + el) = x;
}

// Outputs of one chunk (eight waves), all value columns:
//   o = scale * (Qt (S_r diag e^{b_m})^T + (Qt Kt^T masked) V)
// The gate prefix is scanned in parallel (TPC threads per key channel), the
// masked score block is formed once (ten nonzero 16 x 16 tiles over the
// waves) and kept in LDS in accumulator-pair order, and each wave then owns
// value tiles for IPW token tiles, transposed: O^T = S_r' Qt^T + V^T P^T, with
// rows of S_r read straight from global memory and scaled by e^{b_m} per key
// channel.  V is staged VP columns at a time.
//
// CARRY (bf16, all value columns in one slice): one workgroup walks a group of
// a.group consecutive chunks and reads S_r for the first one only.  Each wave
// holds its value tiles of S_r^T, all key channels, in fp32 accumulators in
// pair order (tile t, row 4 g + r is channel pair_feat(t, g) + r), so that two
// tiles pack into the operand of the output product with 8 consecutive
// channels per lane group.  Per chunk
//   S^T <- S^T diag(e^{b_m})                    (the output's operand)
//   S^T <- diag(e^{b_C - b_m}) (S^T + Kt^T V)   (= e^{b_C} S_r^T + Kd^T V)
// with Kt^T read transposed in the same pair order and V in the matching
// token order; both factors are at most 1.
template <typename T, typename TG, int DK, int VP, int VPW, int IPW, bool CARRY>
__global__ __launch_bounds__(kOutThreads, 1) void gla_out_kernel(const GlaOutArgs a) {
  constexpr int C = kChunk, NT = kOutThreads;
  constexpr int P = Pad<T>::value;
  constexpr int LDQ = DK + P, LDV = VP + P, LDP = C + P, LDB = DK + 4;
  constexpr int NK = DK / 32;
  constexpr int NIG = 4 / IPW, NVG = 8 / NIG;
  static_assert(NVG * NIG == 8 && NVG * VPW * 16 == VP, "wave split");
  constexpr int TPC = NT / DK, TOK = C / TPC;  // scan: threads per channel, tokens per thread
  static_assert(TPC * DK == NT && TOK * TPC == C, "scan split");

  __shared__ __align__(16) T sQt[C * LDQ];
  __shared__ __align__(16) T sKt[C * LDQ];
  // the gates (fp32) share their space with the masked scores and the V slice,
  // both written only once the gates are dead: two workgroups fit on a CU
  constexpr int kBBytes = C * LDB * 4, kPBytes = C * LDP * (int)sizeof(T), kVBytes = C * LDV * (int)sizeof(T);
  __shared__ __align__(16) char sBPV[kBBytes > kPBytes + kVBytes ? kBBytes : kPBytes + kVBytes];
  float* sB = reinterpret_cast<float*>(sBPV);     // gates, then their prefix b
  T* sP = reinterpret_cast<T*>(sBPV);             // masked scores, once sB is dead
  T* sV = reinterpret_cast<T*>(sBPV + kPBytes);   // V slice, once sB is dead
  // e^{b_m}; the same times the decay since the segment began (CARRY: the decay alone)
  __shared__ __align__(16) float sBm[DK], sBe[DK];
  __shared__ __align__(16) float sDc[CARRY ? DK : 4];  // CARRY: e^{b_C - b_m}
  __shared__ float sTot[TPC][DK];
  static_assert(!CARRY || sizeof(T) == 2, "carried state: bf16 path");

  const int N = (a.T + C - 1) / C;
  const int R = CARRY ? a.group : 1, NGR = (N + R - 1) / R;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / NGR, cb = (lb % NGR) * R;
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  const int ce = min((sq.len + C - 1) / C, cb + R);  // a packed sequence's own chunks
  if (cb >= ce) return;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = lane_id();
  const int g4 = l >> 4, c16 = l & 15;
  const int vg = w % NVG, ig = NIG == 1 ? 0 : w / NVG;  // (uniform: no lane-masked branch on the tile)
  const size_t gstride = (size_t)a.H * DK;
  constexpr int NTS = CARRY ? VPW : 1, NPT = CARRY ? 2 * NK : 1;
  f32x4 Sc[NTS][NPT];  // CARRY: this wave's value tiles of S^T, pair order

  // a chunk's q_clean, keys and gates (and, CARRY, values).  CARRY loads each
  // tile of the next chunk as soon as the current chunk is done with its own,
  // so that the loads are in flight while the products run.
  RowTile<T, DK, NT, CARRY> rq, rk;
  RowScales<RowTile<T, DK, NT, CARRY>> fk;  // raw keys: row scales (l2 normalisation)
  RowTile<TG, DK, NT, CARRY> rg;
  RowTile<T, VP, NT, CARRY> rv;
  const Seq sw{(long long)b * a.T, sq.len};  // q_clean: the workspace's padded rows
  auto rows = [&](int c) { return (sq.len - c * C) < C ? (sq.len - c * C) : C; };
  auto load_qk = [&](int c) {
    rq.load(static_cast<const T*>(a.qc) + seq_off(sw, c * C, h, a.H, DK), gstride, rows(c));
    rk.load(static_cast<const T*>(a.k) + seq_off(sq, c * C, h, a.H, DK), gstride, rows(c));
    if (a.rk) fk.load(a.rk + seq_idx(sq, c * C, h, a.H), (size_t)a.H, rows(c));
  };
  auto load_g = [&](int c) { rg.load(static_cast<const TG*>(a.g) + seq_off(sq, c * C, h, a.H, DK), gstride, rows(c)); };
  auto load_v = [&](int c) {
    rv.load(static_cast<const T*>(a.v) + seq_off(sq, c * C, h, a.H, a.dv), (size_t)a.H * a.dv, rows(c));
  };
  if constexpr (CARRY) {
    // S_r of the group's first chunk plus the segment's entry state decayed to
    // it, requested before the chunk's inputs so that the two latencies
    // overlap: lane (g, j) of value tile vt reads channels 32 m + 8 g .. + 7 of
    // value row 16 vt' + j, which are rows 4 g .. 4 g + 3 of tiles 2 m and 2 m + 1
    const int sg0 = a.seg > 0 ? cb / a.seg : 0;
    const bool ent0 = sg0 > 0 && a.entries;
    const T* Sg = static_cast<const T*>(a.states) + ((size_t)bh * N + cb) * a.dv * DK;
    const int NS = a.seg > 0 ? (N + a.seg - 1) / a.seg : 1;
    const T* Eg = static_cast<const T*>(a.entries) + ((size_t)bh * NS + sg0) * a.dv * DK;
    const float* cd = a.cdec + ((size_t)bh * N + cb) * DK;  // decay since the segment began
    Frag<T> fs[VPW][NK], fe[VPW][NK];
    f32x4 de[NK][2];
#pragma unroll
    for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
      for (int m = 0; m < NK; ++m) fs[vt][m] = ld_frag_global(Sg + (size_t)(16 * (vg * VPW + vt)) * DK + 32 * m, (size_t)DK);
    if (ent0) {
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        de[m][0] = *reinterpret_cast<const f32x4*>(cd + 32 * m + 8 * g4);
        de[m][1] = *reinterpret_cast<const f32x4*>(cd + 32 * m + 8 * g4 + 4);
      }
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
        for (int m = 0; m < NK; ++m)
          fe[vt][m] = ld_frag_global(Eg + (size_t)(16 * (vg * VPW + vt)) * DK + 32 * m, (size_t)DK);
    }
    load_g(cb);
    load_qk(cb);
    load_v(cb);
#pragma unroll
    for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        f32x4 x, y;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          x[r] = frag_elem(fs[vt][m], r);
          y[r] = frag_elem(fs[vt][m], 4 + r);
        }
        if (ent0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[r] += frag_elem(fe[vt][m], r) * de[m][0][r];
            y[r] += frag_elem(fe[vt][m], 4 + r) * de[m][1][r];
          }
        }
        Sc[vt][2 * m] = x;
        Sc[vt][2 * m + 1] = y;
      }
  }

  for (int ci = cb; ci < ce; ++ci) {
  // (the barriers of this loop order LDS only: a __syncthreads() fence would
  // also wait for the loads in flight and the output stores)
  if (ci > cb) lds_barrier();  // every wave is done with the previous chunk
  const int r0 = ci * C;
  const int nrow = (sq.len - r0) < C ? (sq.len - r0) : C;
  // past the first segment of the state pass, S_r = local state + the
  // segment's entry state decayed to this chunk (per key channel)
  const int sg = a.seg > 0 ? ci / a.seg : 0;
  const bool ent = sg > 0 && a.entries;

  if constexpr (!CARRY) {
    load_qk(ci);
    load_g(ci);
  }
#pragma unroll
  for (int u = 0; u < RowTile<TG, DK, NT>::NV; ++u) {  // gates as fp32 rows
    const auto x = rg.get(u);
    float* dst = sB + RowTile<TG, DK, NT>::row(u) * LDB + RowTile<TG, DK, NT>::col(u);
    *reinterpret_cast<f32x4*>(dst) = f32x4{f32(x[0]), f32(x[1]), f32(x[2]), f32(x[3])};
    *reinterpret_cast<f32x4*>(dst + 4) = f32x4{f32(x[4]), f32(x[5]), f32(x[6]), f32(x[7])};
  }
  if constexpr (CARRY)
    if (ci + 1 < ce) load_g(ci + 1);
  lds_barrier();
  {  // inclusive prefix over the chunk, TPC threads per channel
    const int c = tid % DK, part = tid / DK, j0 = part * TOK;
    float x[TOK];
#pragma unroll
    for (int j = 0; j < TOK; ++j) x[j] = sB[(j0 + j) * LDB + c];
#pragma unroll
    for (int j = 1; j < TOK; ++j) x[j] += x[j - 1];
    sTot[part][c] = x[TOK - 1];
    lds_barrier();
    float off = 0.f;
#pragma unroll
    for (int p2 = 0; p2 < TPC - 1; ++p2)
      if (p2 < part) off += sTot[p2][c];
#pragma unroll
    for (int j = 0; j < TOK; ++j) sB[(j0 + j) * LDB + c] = x[j] + off;
    if (j0 <= C / 2 - 1 && C / 2 - 1 < j0 + TOK) {
      const float bm = __expf(x[C / 2 - 1 - j0] + off);
      sBm[c] = bm;
      if (!CARRY && ent) sBe[c] = bm * a.cdec[((size_t)bh * N + ci) * DK + c];
    }
  }
  lds_barrier();
  if (CARRY && tid < DK) sDc[tid] = __expf(sB[(C - 1) * LDB + tid] - sB[(C / 2 - 1) * LDB + tid]);
  if (a.rk) fk.apply(rk);
  // Qt = q e^{b - b_m}, Kt = k e^{b_m - b}
#pragma unroll
  for (int u = 0; u < RowTile<T, DK, NT>::NV; ++u) {
    const int j = RowTile<T, DK, NT>::row(u), cc = RowTile<T, DK, NT>::col(u);
    const auto xq = rq.get(u), xk = rk.get(u);
    typename RowTile<T, DK, NT>::vec_t qo, ko;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float d = sB[j * LDB + cc + e] - sB[(C / 2 - 1) * LDB + cc + e];
      qo[e] = to<T>(f32(xq[e]) * __expf(d));
      ko[e] = to<T>(f32(xk[e]) * __expf(-d));
    }
    *reinterpret_cast<typename RowTile<T, DK, NT>::vec_t*>(sQt + j * LDQ + cc) = qo;
    *reinterpret_cast<typename RowTile<T, DK, NT>::vec_t*>(sKt + j * LDQ + cc) = ko;
  }
  if constexpr (CARRY)
    if (ci + 1 < ce) load_qk(ci + 1);
  lds_barrier();  // sB is dead from here on

  // masked score tiles, transposed (row j, column i), stored as rows i
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
    store4(sP + i * LDP + acc_pos(16 * J + 4 * g4), x[0], x[1], x[2], x[3]);
  }

  const T* Sg = static_cast<const T*>(a.states) + ((size_t)bh * N + ci) * a.dv * DK;
  const int NS = a.seg > 0 ? (N + a.seg - 1) / a.seg : 1;
  const T* Eg = ent ? static_cast<const T*>(a.entries) + ((size_t)bh * NS + sg) * a.dv * DK : nullptr;
  T* o = static_cast<T*>(a.o);
  if constexpr (CARRY) {
    rv.store(sV, LDV);
    if (ci + 1 < ce) load_v(ci + 1);
    // S^T diag(e^{b_m}) in place, the output's operand
#pragma unroll
    for (int m = 0; m < NK; ++m) {
      const f32x4 e0 = *reinterpret_cast<const f32x4*>(sBm + 32 * m + 8 * g4);
      const f32x4 e1 = *reinterpret_cast<const f32x4*>(sBm + 32 * m + 8 * g4 + 4);
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) {
        Sc[vt][2 * m] *= e0;
        Sc[vt][2 * m + 1] *= e1;
      }
    }
    lds_barrier();  // sV and sP are ready
    // V in the token order of the accumulator pairs (for both products)
    Frag<T> vf[VPW][2];
#pragma unroll
    for (int vt = 0; vt < VPW; ++vt)
#pragma unroll
      for (int kq = 0; kq < 2; ++kq) vf[vt][kq] = ld_frag_tr_acc(sV + 32 * kq * LDV + 16 * (vg * VPW + vt), LDV);
#pragma unroll
    for (int it = 0; it < IPW; ++it) {
      const int I = ig * IPW + it;
      const int i = 16 * I + c16;
      f32x4 acc[VPW];
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) acc[vt] = zero4();
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        const Frag<T> qf = ld_frag(sQt + 16 * I * LDQ + 32 * m, LDQ);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) mma(acc[vt], acc_pair_frag<T>(Sc[vt][2 * m], Sc[vt][2 * m + 1]), qf);
      }
      const Frag<T> pf0 = ld_frag(sP + 16 * I * LDP, LDP);
      const Frag<T> pf1 = ld_frag(sP + 16 * I * LDP + 32, LDP);
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) {
        const int vl = 16 * (vg * VPW + vt);
        mma(acc[vt], vf[vt][0], pf0);
        if (I >= 2) mma(acc[vt], vf[vt][1], pf1);  // keys 32..63 precede row i
        if (i < nrow)
          store4(o + seq_off(sq, r0 + i, h, a.H, a.dv) + vl + 4 * g4, a.scale * acc[vt][0], a.scale * acc[vt][1],
                 a.scale * acc[vt][2], a.scale * acc[vt][3]);
      }
    }
    if (ci + 1 < ce) {
      // S^T <- diag(e^{b_C - b_m}) (S^T + Kt^T V), per 32-channel block
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        Frag<T> kf[2][2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int kq = 0; kq < 2; ++kq) kf[hh][kq] = ld_frag_tr_acc_pair(sKt + 32 * kq * LDQ, LDQ, 2 * m + hh);
        const f32x4 d0 = *reinterpret_cast<const f32x4*>(sDc + 32 * m + 8 * g4);
        const f32x4 d1 = *reinterpret_cast<const f32x4*>(sDc + 32 * m + 8 * g4 + 4);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) {
#pragma unroll
          for (int kq = 0; kq < 2; ++kq) {
            mma(Sc[vt][2 * m], kf[0][kq], vf[vt][kq]);
            mma(Sc[vt][2 * m + 1], kf[1][kq], vf[vt][kq]);
          }
          Sc[vt][2 * m] *= d0;
          Sc[vt][2 * m + 1] *= d1;
        }
      }
    }
  } else
  for (int vp = 0; vp < a.dv; vp += VP) {
    if (vp > 0) lds_barrier();  // every wave is done with the previous V slice
    {
      RowTile<T, VP, NT> rv;
      rv.load(static_cast<const T*>(a.v) + seq_off(sq, r0, h, a.H, a.dv) + vp, (size_t)a.H * a.dv, nrow);
      rv.store(sV, LDV);
    }
    // this wave's rows of S_r (k = key channel), scaled by e^{b_m}
    Frag<T> sfr[VPW][NK];
#pragma unroll
    for (int vt = 0; vt < VPW; ++vt) {
      const int vr = vp + 16 * (vg * VPW + vt);
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        Frag<T> f = ld_frag_global(Sg + (size_t)vr * DK + 32 * m, (size_t)DK);
        const f32x4 e0 = *reinterpret_cast<const f32x4*>(sBm + 32 * m + 8 * g4);
        const f32x4 e1 = *reinterpret_cast<const f32x4*>(sBm + 32 * m + 8 * g4 + 4);
        if (ent) {
          const Frag<T> fe = ld_frag_global(Eg + (size_t)vr * DK + 32 * m, (size_t)DK);
          const f32x4 d0 = *reinterpret_cast<const f32x4*>(sBe + 32 * m + 8 * g4);
          const f32x4 d1 = *reinterpret_cast<const f32x4*>(sBe + 32 * m + 8 * g4 + 4);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            set_frag_elem(f, e, frag_elem(f, e) * (e < 4 ? e0[e] : e1[e - 4]) + frag_elem(fe, e) * (e < 4 ? d0[e] : d1[e - 4]));
        } else if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int e = 0; e < 8; ++e) f.v[e] = to<T>(f32(f.v[e]) * (e < 4 ? e0[e] : e1[e - 4]));
        } else {
          f.lo *= e0;
          f.hi *= e1;
        }
        sfr[vt][m] = f;
      }
    }
    lds_barrier();  // sV and sP are ready
#pragma unroll
    for (int it = 0; it < IPW; ++it) {
      const int I = ig * IPW + it;
      const int i = 16 * I + c16;
      // S_r' Qt^T one k step at a time (one q fragment live), all value tiles
      f32x4 acc[VPW];
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) acc[vt] = zero4();
#pragma unroll
      for (int m = 0; m < NK; ++m) {
        const Frag<T> qf = ld_frag(sQt + 16 * I * LDQ + 32 * m, LDQ);
#pragma unroll
        for (int vt = 0; vt < VPW; ++vt) mma(acc[vt], sfr[vt][m], qf);
      }
      const Frag<T> pf0 = ld_frag(sP + 16 * I * LDP, LDP);
      const Frag<T> pf1 = ld_frag(sP + 16 * I * LDP + 32, LDP);
#pragma unroll
      for (int vt = 0; vt < VPW; ++vt) {
        const int vl = 16 * (vg * VPW + vt);  // value column within the slice
        mma(acc[vt], ld_frag_tr_acc(sV + vl, LDV), pf0);
        if (I >= 2) mma(acc[vt], ld_frag_tr_acc(sV + 32 * LDV + vl, LDV), pf1);  // keys 32..63 precede row i
        if (i < nrow)
          store4(o + seq_off(sq, r0 + i, h, a.H, a.dv) + vp + vl + 4 * g4, a.scale * acc[vt][0],
                 a.scale * acc[vt][1], a.scale * acc[vt][2], a.scale * acc[vt][3]);
      }
    }
  }
  }  // chunks of the group
}

namespace {
int gla_nseg(const GlaStateArgs& a) {
  const int N = (a.T + kChunk - 1) / kChunk;
  return a.seg > 0 ? (N + a.seg - 1) / a.seg : 1;
}
template <typename T, typename TG, int NVT, bool kRev>
hipError_t run_gla_state_v(const GlaStateArgs& a, hipStream_t st) {
  const int nblk = a.B * a.H * (a.dk / 64) * (a.dv / (16 * NVT)) * gla_nseg(a);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_state_kernel<T, TG, NVT, kRev>), dim3(nblk), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}
// 64-wide value slices when they still give every SIMD a wave, else 32 or 16.
template <typename T, typename TG, bool kRev = false>
hipError_t run_gla_state(const GlaStateArgs& a, hipStream_t st) {
  const long long waves64 = (long long)a.B * a.H * (a.dk / 64) * (a.dv / 64) * 4 * gla_nseg(a);
  if (waves64 >= 1024) return run_gla_state_v<T, TG, 4, kRev>(a, st);
  if (waves64 * 2 >= 1024) return run_gla_state_v<T, TG, 2, kRev>(a, st);
  return run_gla_state_v<T, TG, 1, kRev>(a, st);
}
template <typename T, typename TG, int DK, int VP, int VPW, int IPW>
hipError_t run_gla_out_v(const GlaOutArgs& a, hipStream_t st) {
  const int N = (a.T + kChunk - 1) / kChunk;
  if constexpr (sizeof(T) == 2) {
    if (a.group > 1) {
      if (a.dv != VP) return hipErrorInvalidValue;  // the carried state covers every value column
      const int nblk = a.B * a.H * ((N + a.group - 1) / a.group);
      if (nblk == 0) return hipSuccess;
      hipLaunchKernelGGL((gla_out_kernel<T, TG, DK, VP, VPW, IPW, true>), dim3(nblk), dim3(kOutThreads), 0, st, a);
      return hipGetLastError();
    }
  }
  const int nblk = a.B * a.H * N;
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((gla_out_kernel<T, TG, DK, VP, VPW, IPW, false>), dim3(nblk), dim3(kOutThreads), 0, st, a);
  return hipGetLastError();
}
// V is staged at most 256 columns (fp32: 128) at a time.
template <typename T, typename TG, int DK>
hipError_t run_gla_out_dk(const GlaOutArgs& a, hipStream_t st) {
  constexpr bool kWide = sizeof(T) == 2;
  switch (a.dv) {
    case 64: return run_gla_out_v<T, TG, DK, 64, 1, 2>(a, st);
    case 128: return run_gla_out_v<T, TG, DK, 128, 1, 4>(a, st);
    default:
      if constexpr (kWide) return run_gla_out_v<T, TG, DK, 256, 2, 4>(a, st);
      else return run_gla_out_v<T, TG, DK, 128, 1, 4>(a, st);
  }
}
template <typename T, typename TG>
hipError_t run_gla_out(const GlaOutArgs& a, hipStream_t st) {
  if (a.dk == 64) return run_gla_out_dk<T, TG, 64>(a, st);
  if (a.dk == 128) return run_gla_out_dk<T, TG, 128>(a, st);
  return hipErrorInvalidValue;
}
}  // namespace

int gla_out_group(int B, int H, int T, int dk, int dv, bool is_bf16) {
  // The carried form needs every value column in one staged slice (bf16:
  // dv <= 256).  A group of G chunks takes a compute unit and costs about
  // G + 1 chunk steps (the stored state read once); a workgroup of the
  // one-chunk form (two per compute unit) about 3, its state read and the
  // state pass's store of every chunk included.  The G of least rounds x cost
  // wins, the largest on a tie.  Measured per call: T = 2048 with 32 heads
  // 142 us (one chunk each), 128 (G = 2), 118.5 (4), 140 (8); T = 20480 with 4
  // heads 203, 188.5, 192, 185.
  if (!is_bf16 || dv > 256 || (dk != 64 && dk != 128)) return 1;
  const long long bh = (long long)B * H;
  const long long N = (T + kChunk - 1) / kChunk;
  int best = 1;
  long long best_cost = ((bh * N + 511) / 512) * 3;
  for (int g = 2; g <= 8; g *= 2) {
    const long long rounds = (bh * ((N + g - 1) / g) + 255) / 256;
    const long long cost = rounds * (g + 1);
    if (cost <= best_cost) {
      best_cost = cost;
      best = g;
    }
  }
  return best;
}

bool gla_supported(int dk, int dv, bool is_bf16) {
  const bool dv_ok = dv == 64 || dv == 128 || dv == 256 || dv == 512;
  (void)is_bf16;
  return dv_ok && (dk == 64 || dk == 128);
}

hipError_t launch_gla_state(const GlaStateArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? run_gla_state<bf16_t, bf16_t>(a, st) : run_gla_state<bf16_t, float>(a, st);
  return gate_bf16 ? run_gla_state<float, bf16_t>(a, st) : run_gla_state<float, float>(a, st);
}

// The training step's reverse state scan (kRev), one segment.
hipError_t launch_gla_dstate(const DstateArgs& d, bool is_bf16, bool gate_bf16, hipStream_t st) {
  GlaStateArgs a{};
  a.k = d.qc;
  a.v = d.dO;
  a.g = d.g;
  a.states = d.dstates;
  a.B = d.B;
  a.T = d.T;
  a.H = d.H;
  a.dk = d.dk;
  a.dv = d.dv;
  a.scale = d.scale;
  if (is_bf16) return gate_bf16 ? run_gla_state<bf16_t, bf16_t, true>(a, st) : run_gla_state<bf16_t, float, true>(a, st);
  return gate_bf16 ? run_gla_state<float, bf16_t, true>(a, st) : run_gla_state<float, float, true>(a, st);
}

hipError_t launch_gla_scan(const GlaScanArgs& a, bool is_bf16, hipStream_t st) {
  const long long n4 = (long long)a.B * a.H * a.dv * a.dk / 4;
  if (n4 == 0) return hipSuccess;
  const unsigned nblk = (unsigned)((n4 + 255) / 256);
  if (is_bf16) hipLaunchKernelGGL((gla_scan_kernel<bf16_t>), dim3(nblk), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((gla_scan_kernel<float>), dim3(nblk), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gla_out(const GlaOutArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16) return gate_bf16 ? run_gla_out<bf16_t, bf16_t>(a, st) : run_gla_out<bf16_t, float>(a, st);
  return gate_bf16 ? run_gla_out<float, bf16_t>(a, st) : run_gla_out<float, float>(a, st);
}

}  // namespace ccq
