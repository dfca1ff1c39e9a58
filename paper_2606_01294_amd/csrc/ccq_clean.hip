// ccq_clean.hip -- CCQ query contraction (Eq. clean), chunkwise (App. B,
// Alg. 1).  For token t (1-based position t = t0 + index + 1):
//
//   Sigma_t   = Cbar_t - mu_t mu_t^T,  Cbar_t = (1/t) sum_{j<=t} k_j k_j^T,
//   mu_t      = m_t / t,               m_t    = sum_{j<=t} k_j
//   q_clean_t = q_t - lambda_t Sigma_t q_t
//
// Sigma_t is unchanged when every key is shifted by one vector c, which this
// file uses to keep bf16 products well conditioned when the keys share a
// large common mean:
//
//   t Sigma_t q = sum_{j<=t} (k_j - c)(k_j - c)^T q - (m'_t . q) m'_t / t,
//   m'_t = m_t - t c.
//
// The sequence is cut into segments of `seg` chunks and c = c_s is the mean
// key of segment s.  For token i of chunk r in segment s:
//
//   t_i Sigma q_i = S'_s q_i + sum_{j in s, j<=i} (q_i . k'_j) k'_j - (cq'_i / t_i) m'_i
//   S'_s  = sum_{j before s} (k_j - c_s)(k_j - c_s)^T      (entry second moment)
//   k'_j  = k_j - c_s,  cq'_i = m'_i . q_i
//
// Three kernels:
//   clean_gram    raw sums of k k^T per segment, and of k per chunk and segment
//   clean_prefix  S'_s by a prefix over segments (fp32), stored in io dtype
//   clean_out     one workgroup per chunk pair: S'_s q plus the causal product
//                 over the segment's centred keys, all in MFMA tiles
// Without centring (Sigma = Cbar) the same kernels run with c_s = 0 and no
// mean terms.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {
namespace {

__host__ __device__ inline int n_chunks(int T) { return (T + kChunk - 1) / kChunk; }
__host__ __device__ inline int n_segs(int T, int seg) { return (n_chunks(T) + seg - 1) / seg; }

template <typename T>
__device__ __forceinline__ f32x4 load4f(const T* p) {
  if constexpr (sizeof(T) == 2) {
    const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
    return f32x4{f32(v[0]), f32(v[1]), f32(v[2]), f32(v[3])};
  } else {
    return *reinterpret_cast<const f32x4*>(p);
  }
}

}  // namespace

// Raw segment Gram matrix G_s = sum_{j in s} k_j k_j^T, one workgroup per
// (head, segment); wave w owns rows [w RW, (w+1) RW) and all columns, so each
// chunk of keys is read from memory once.  The chunk and segment key sums come
// from the same products (a ones column).  G is symmetric: each tile is
// written transposed, as rows of four consecutive features (16-byte stores).
template <typename T, int DK>
__global__ __launch_bounds__(64 * (DK >= 128 ? 8 : 4), 1) void clean_gram_kernel(const CleanArgs a) {
  constexpr int C = kChunk, P = Pad<T>::value, LDK = DK + P;
  constexpr int NWG = DK >= 128 ? 8 : 4, NTG = 64 * NWG;
  constexpr int RW = DK / NWG;  // rows per wave
  constexpr int RT = RW / 16;   // row tiles per wave
  constexpr int CT = DK / 16;   // column tiles
  __shared__ __align__(16) T sK[2][C * LDK];

  const int NC = n_chunks(a.T), NS = n_segs(a.T, a.seg);
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / NS, s = lb % NS;
  const int b = bh / a.H, h = bh % a.H;
  const int w = wave_id(), l = lane_id(), g4 = l >> 4, c16 = l & 15;
  const int a0 = w * RW;
  const T* k = static_cast<const T*>(a.k);
  const size_t gstride = (size_t)a.H * DK;
  const int cbeg = s * a.seg, cend = min(NC, cbeg + a.seg);

  f32x4 acc[RT][CT], stot[RT];
#pragma unroll
  for (int v = 0; v < RT; ++v) {
    stot[v] = zero4();
#pragma unroll
    for (int t = 0; t < CT; ++t) acc[v][t] = zero4();
  }

  RowTile<T, DK, NTG> rk;
  auto load = [&](int c) {
    rk.load(k + tok_off(b, c * C, h, a.T, a.H, DK), gstride, min(C, a.T - c * C));
  };
  load(cbeg);
  const Frag<T> ones = ones_col_frag<T>();

  for (int c = cbeg; c < cend; ++c) {
    T* buf = sK[(c - cbeg) & 1];  // the other buffer may still be read by a slower wave
    rk.store(buf, LDK);
    if (c + 1 < cend) load(c + 1);
    __syncthreads();
    f32x4 msum[RT];
#pragma unroll
    for (int v = 0; v < RT; ++v) msum[v] = zero4();
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 32) {
      Frag<T> fa[RT];
#pragma unroll
      for (int v = 0; v < RT; ++v) {
        fa[v] = ld_frag_tr(buf + k0 * LDK + a0 + 16 * v, LDK);
        mma(msum[v], fa[v], ones);
      }
#pragma unroll
      for (int t = 0; t < CT; ++t) {
        const Frag<T> fb = ld_frag_tr(buf + k0 * LDK + 16 * t, LDK);
#pragma unroll
        for (int v = 0; v < RT; ++v) mma(acc[v][t], fa[v], fb);
      }
    }
    if (c16 == 0) {
#pragma unroll
      for (int v = 0; v < RT; ++v) {
        stot[v] += msum[v];
        *reinterpret_cast<f32x4*>(a.csum + ((size_t)bh * NC + c) * DK + a0 + 16 * v + 4 * g4) = msum[v];
      }
    }
  }
  if (c16 == 0) {
#pragma unroll
    for (int v = 0; v < RT; ++v)
      *reinterpret_cast<f32x4*>(a.ssum + ((size_t)bh * NS + s) * DK + a0 + 16 * v + 4 * g4) = stot[v];
  }
  // acc[v][t][r] = G[a0 + 16 v + 4 g4 + r][16 t + c16], stored at the mirror position
  float* G = a.gram + ((size_t)bh * NS + s) * DK * DK;
#pragma unroll
  for (int v = 0; v < RT; ++v)
#pragma unroll
    for (int t = 0; t < CT; ++t)
      *reinterpret_cast<f32x4*>(G + (size_t)(16 * t + c16) * DK + a0 + 16 * v + 4 * g4) = acc[v][t];
}

// S'_s = S_s - M'_s c_s^T - c_s M'_s^T - n_s c_s c_s^T with S_s the raw second
// moment before segment s (prefix of the Gram matrices, fp32), c_s the mean
// key of segment s, n_s the tokens before it and M'_s = M_s - n_s c_s the key
// sum before it about c_s (running sums of the segment key sums, kept for this
// thread's row and four columns); four elements per thread.  S'_s is stored in
// 64-column slices, each a contiguous [dk][64] block.  Also the final Cbar_T
// and mu_T.
template <typename T, int DK>
__global__ __launch_bounds__(256) void clean_prefix_kernel(const CleanArgs a) {
  constexpr int PER = DK * DK / 4 / 256;  // workgroups per head
  const int bh = blockIdx.x / PER;
  const int e = ((blockIdx.x % PER) * 256 + threadIdx.x) * 4;
  const int ra = e / DK, cb = e % DK;
  const int NC = n_chunks(a.T), NS = n_segs(a.T, a.seg);
  const float t0f = (float)a.t0;
  f32x4 acc = zero4();
  if (a.C0) acc = *reinterpret_cast<const f32x4*>(a.C0 + ((size_t)bh * DK + ra) * DK + cb) * t0f;
  float run_a = a.mu0 ? t0f * a.mu0[(size_t)bh * DK + ra] : 0.f;  // raw key sums before s
  f32x4 run_b = a.mu0 ? *reinterpret_cast<const f32x4*>(a.mu0 + (size_t)bh * DK + cb) * t0f : zero4();
  T* Sp = static_cast<T*>(a.sprime);
  for (int s = 0; s < NS; ++s) {
    const size_t so = (size_t)bh * NS + s;
    const int cbeg = s * a.seg, cend = min(NC, cbeg + a.seg);
    const float len = (float)(min(a.T, cend * kChunk) - cbeg * kChunk);
    const float ns = t0f + (float)((int64_t)cbeg * kChunk);
    const float tot_a = a.ssum[so * DK + ra];
    const f32x4 tot_b = *reinterpret_cast<const f32x4*>(a.ssum + so * DK + cb);
    const f32x4 g = *reinterpret_cast<const f32x4*>(a.gram + (so * DK + ra) * DK + cb);
    const float ca = a.centered ? tot_a / len : 0.f;
    const f32x4 cb4 = a.centered ? tot_b / len : zero4();
    const float ma = run_a - ns * ca;
    const f32x4 mb4 = run_b - ns * cb4;
    f32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = acc[q] - ma * cb4[q] - ca * mb4[q] - ns * ca * cb4[q];
    store4(Sp + so * DK * DK + ((size_t)(cb >> 6) * DK + ra) * 64 + (cb & 63), o[0], o[1], o[2], o[3]);
    acc += g;
    run_a += tot_a;
    run_b += tot_b;
  }
  const float inv = 1.f / (t0f + (float)a.T);
  if (a.CT) *reinterpret_cast<f32x4*>(a.CT + ((size_t)bh * DK + ra) * DK + cb) = acc * inv;
  if (a.muT && ra == 0) *reinterpret_cast<f32x4*>(a.muT + (size_t)bh * DK + cb) = run_b * inv;
}

// One workgroup per CPW consecutive chunks of a segment; wave w owns rows
// i = 16 (w % 4) .. + 15 of chunk w / 4.  All products are kept transposed
// (output feature n in the accumulator row, token i in its column) so that
// score tiles feed the next product from registers:
//   acc^T  = S'_s x^T               (S' staged through LDS one 64-column slice
//                                     at a time, double-buffered)
//   sc^T   = K'_blk x^T,  acc^T += K'_blk^T sc^T        (each block of the segment)
// The slice buffers are reused for the key blocks, and both are shared by the
// CPW chunks, which halves (CPW = 2) the global round trips per chunk.
// On the diagonal block the scores are masked to j <= i and shifted by
// -cq'_i / t_i, which folds the within-chunk part of m'_i into the product.
template <typename T, int DK, int CPW>
__global__ __launch_bounds__(kThreads * CPW, 1) void clean_out_kernel(const CleanArgs a) {
  constexpr int C = kChunk, P = Pad<T>::value, LDK = DK + P, LDP = 64 + P;
  constexpr int NT = kThreads * CPW;
  constexpr int NK = DK / 32, NN = DK / 16, NP = DK / 64;
  constexpr int BUF = (DK * LDP > C * LDK) ? DK * LDP : C * LDK;  // elements per buffer
  constexpr int NVS = DK * 64 / 8 / NT;                            // slice vectors per thread
  static_assert(NVS >= 1 && DK * 64 % (8 * NT) == 0, "slice split");
  typedef typename RowTile<T, DK, NT>::vec_t vec_t;
  __shared__ __align__(16) T sbuf[2 * BUF];
  __shared__ __align__(16) float sC[DK], sMs[DK], sMr[CPW][DK];

  const int NC = n_chunks(a.T), NS = n_segs(a.T, a.seg);
  const int NG = (NC + CPW - 1) / CPW;
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / NG, ch0 = (lb % NG) * CPW;
  const int chl = min(NC - 1, ch0 + CPW - 1);  // last chunk of the group
  const int b = bh / a.H, h = bh % a.H;
  const int s = ch0 / a.seg, cbeg = s * a.seg;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id(), g4 = l >> 4, c16 = l & 15;
  const int wr = w & 3, ch = ch0 + (w >> 2);
  const bool has = ch < NC;  // this wave's chunk exists
  const int r0 = ch * C, nrow = has ? min(C, a.T - r0) : 0;
  const T* x = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  const size_t gstride = (size_t)a.H * DK;
  const float t0f = (float)a.t0;
  const size_t so = (size_t)bh * NS + s;

  // this wave's rows of x as B fragments (column = token); rows past the end
  // repeat the last row and are never written back
  const int i = 16 * wr + c16;
  const bool iok = i < nrow;
  Frag<T> qf[NK];
  {
    const int row = has ? r0 + (iok ? i : nrow - 1) : 0;
    const T* xr = x + tok_off(b, row, h, a.T, a.H, DK) + 8 * g4;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      if constexpr (sizeof(T) == 2) {
        qf[kk].v = *reinterpret_cast<const bf16x8*>(xr + 32 * kk);
      } else {
        qf[kk].lo = *reinterpret_cast<const f32x4*>(xr + 32 * kk);
        qf[kk].hi = *reinterpret_cast<const f32x4*>(xr + 32 * kk + 4);
      }
    }
  }
  RowTile<T, DK, NT> rk;
  auto load_block = [&](int c) {
    rk.load(k + tok_off(b, c * C, h, a.T, a.H, DK), gstride, min(C, a.T - c * C));
  };
  load_block(cbeg);
  // key statistics of the segment, one thread per feature: the centre c_s, the
  // key sum before the segment about c_s (M'_s) and before each of this
  // group's chunks (M'_r), from the segment and chunk key sums
  for (int d = tid; d < DK; d += NT) {
    const float* ss = a.ssum + (size_t)bh * NS * DK + d;
    float run = a.mu0 ? t0f * a.mu0[(size_t)bh * DK + d] : 0.f;
#pragma unroll 8
    for (int p = 0; p < s; ++p) run += ss[(size_t)p * DK];
    const int cend = min(NC, cbeg + a.seg);
    const float len = (float)(min(a.T, cend * C) - cbeg * C);
    const float cen = a.centered ? ss[(size_t)s * DK] / len : 0.f;
    float mp = run - (t0f + (float)(cbeg * C)) * cen;
    sC[d] = cen;
    sMs[d] = mp;
    const float* cs = a.csum + (size_t)bh * NC * DK + d;
    for (int c = cbeg; c <= chl; ++c) {
      if (c >= ch0) sMr[c - ch0][d] = mp;
      mp += cs[(size_t)c * DK] - (float)min(C, a.T - c * C) * cen;
    }
  }

  // entry term S'_s x_i, one 64-column slice of S' per step
  f32x4 acc[NN];
#pragma unroll
  for (int tn = 0; tn < NN; ++tn) acc[tn] = zero4();
  {
    // all slices are requested up front when they fit in registers (the whole
    // of S' is DK * DK / 8 / NT vectors per thread), else one slice ahead
    constexpr bool kAll = NVS * NP <= 16;
    constexpr int NB = kAll ? NP : 2;
    const T* sp = static_cast<const T*>(a.sprime) + so * DK * DK;
    vec_t ps[NB][NVS];
    auto load_slice = [&](int p) {
#pragma unroll
      for (int u = 0; u < NVS; ++u)
        ps[kAll ? p : (p & 1)][u] =
            *reinterpret_cast<const vec_t*>(sp + (size_t)p * DK * 64 + (size_t)(tid + NT * u) * 8);
    };
    if constexpr (kAll) {
#pragma unroll
      for (int p = 0; p < NP; ++p) load_slice(p);
    } else {
      load_slice(0);
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      T* pb = sbuf + (p & 1) * BUF;
#pragma unroll
      for (int u = 0; u < NVS; ++u) {
        const int e = tid + NT * u;
        *reinterpret_cast<vec_t*>(pb + (e >> 3) * LDP + 8 * (e & 7)) = ps[kAll ? p : (p & 1)][u];
      }
      if (!kAll && p + 1 < NP) load_slice(p + 1);
      __syncthreads();  // (also publishes sC, sMs, sMr)
      if (has) {
#pragma unroll
        for (int tn = 0; tn < NN; ++tn) {
          mma(acc[tn], ld_frag(pb + 16 * tn * LDP, LDP), qf[2 * p]);
          mma(acc[tn], ld_frag(pb + 16 * tn * LDP + 32, LDP), qf[2 * p + 1]);
        }
      }
    }
  }

  // M'_s . x_i and c_s . x_i (each lane holds 8 features per k step)
  float mq = 0.f, cx = 0.f;
#pragma unroll
  for (int kk = 0; kk < NK; ++kk)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = 32 * kk + 8 * g4 + e;
      const float xv = frag_elem(qf[kk], e);
      mq += xv * sMs[d];
      cx += xv * sC[d];
    }
  mq += __shfl_xor(mq, 16);
  mq += __shfl_xor(mq, 32);
  cx += __shfl_xor(cx, 16);
  cx += __shfl_xor(cx, 32);

  const float ti = t0f + (float)(r0 + i + 1);
  float rs = 0.f, cqp = 0.f;
  for (int jb = cbeg; jb <= chl; ++jb) {
    T* buf = sbuf + ((NP + jb - cbeg) & 1) * BUF;
    // centred keys of block jb; the other buffer may still be read by a wave
    // working on the step before, this one was released by the last barrier
#pragma unroll
    for (int u = 0; u < RowTile<T, DK, NT>::NV; ++u) {
      const vec_t kv = rk.get(u);
      const int col = RowTile<T, DK, NT>::col(u);
      vec_t y;
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = to<T>(f32(kv[e]) - sC[col + e]);
      *reinterpret_cast<vec_t*>(buf + RowTile<T, DK, NT>::row(u) * LDK + col) = y;
    }
    if (jb < chl) load_block(jb + 1);
    __syncthreads();
    if (!has || jb > ch) continue;  // wave-uniform: this chunk's window has ended

    const bool diag = jb == ch;
    f32x4 sc[4];
#pragma unroll
    for (int J = 0; J < 4; ++J) {
      sc[J] = zero4();
      if (!diag || J <= wr)
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) mma(sc[J], ld_frag(buf + 16 * J * LDK + 32 * kk, LDK), qf[kk]);
    }
    if (diag) {
#pragma unroll
      for (int J = 0; J < 4; ++J)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (16 * J + 4 * g4 + r > i) sc[J][r] = 0.f;
    }
#pragma unroll
    for (int J = 0; J < 4; ++J) rs += sc[J][0] + sc[J][1] + sc[J][2] + sc[J][3];
    if (diag) {
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      cqp = mq + rs;  // m'_i . x_i
      if (a.centered) {
        const float sub = cqp / ti;
#pragma unroll
        for (int J = 0; J < 4; ++J)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * J + 4 * g4 + r <= i) sc[J][r] -= sub;
      }
    }
    const Frag<T> f0 = acc_pair_frag<T>(sc[0], sc[1]);
    const Frag<T> f1 = acc_pair_frag<T>(sc[2], sc[3]);
    const bool upper = !diag || wr >= 2;  // keys 32..63 can precede row i
#pragma unroll
    for (int tn = 0; tn < NN; ++tn) {
      mma(acc[tn], ld_frag_tr_acc(buf + 16 * tn, LDK), f0);
      if (upper) mma(acc[tn], ld_frag_tr_acc(buf + 32 * LDK + 16 * tn, LDK), f1);
    }
  }

  if (!iok) return;
  // epilogue: every load is issued before the first store, and the optional
  // outputs are written in loops of their own, so the loads and stores of the
  // NN tiles overlap instead of forming NN round trips to memory
  const float inv = 1.f / ti;
  const float lam = a.lam[((size_t)b * a.T + r0 + i) * a.H + h];
  const float msub = a.centered ? cqp * inv : 0.f;
  const size_t rowoff = tok_off(b, r0 + i, h, a.T, a.H, DK) + 4 * g4;
  const float* mrow = sMr[w >> 2] + 4 * g4;
  f32x4 xb[NN];
  if (a.base) {
#pragma unroll
    for (int tn = 0; tn < NN; ++tn) xb[tn] = *reinterpret_cast<const f32x4*>(a.base + rowoff + 16 * tn);
  } else {
#pragma unroll
    for (int tn = 0; tn < NN; ++tn) xb[tn] = load4f(x + rowoff + 16 * tn);
  }
#pragma unroll
  for (int tn = 0; tn < NN; ++tn) {  // acc <- Sigma_t x_t (the correction before lambda)
    const f32x4 mr = *reinterpret_cast<const f32x4*>(mrow + 16 * tn);
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[tn][r] = (acc[tn][r] - msub * mr[r]) * inv;
  }
  T* qc = static_cast<T*>(a.qclean);
#pragma unroll
  for (int tn = 0; tn < NN; ++tn) {
    f32x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = xb[tn][r] - lam * acc[tn][r];
    store4(qc + rowoff + 16 * tn, o[0], o[1], o[2], o[3]);
    xb[tn] = o;
  }
  if (a.qclean_dbg) {
#pragma unroll
    for (int tn = 0; tn < NN; ++tn) *reinterpret_cast<f32x4*>(a.qclean_dbg + rowoff + 16 * tn) = xb[tn];
  }
  if (a.corr) {
#pragma unroll
    for (int tn = 0; tn < NN; ++tn) *reinterpret_cast<f32x4*>(a.corr + rowoff + 16 * tn) = acc[tn];
  }
  if (a.mdot && g4 == 0) a.mdot[((size_t)b * a.T + r0 + i) * a.H + h] = cqp + ti * cx;  // raw m . x
}

namespace {
template <typename T, int DK>
hipError_t run_gram(const CleanArgs& a, hipStream_t st) {
  const long long nblk = (long long)a.B * a.H * n_segs(a.T, a.seg);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((clean_gram_kernel<T, DK>), dim3((unsigned)nblk), dim3(64 * (DK >= 128 ? 8 : 4)), 0,
                     st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_prefix(const CleanArgs& a, hipStream_t st) {
  const long long nblk = (long long)a.B * a.H * (DK * DK / 1024);
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL((clean_prefix_kernel<T, DK>), dim3((unsigned)nblk), dim3(256), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_out(const CleanArgs& a, hipStream_t st) {
  const int nc = n_chunks(a.T);
  if ((long long)a.B * a.H * nc == 0) return hipSuccess;
  if (nc >= 2 && a.seg % 2 == 0) {  // two chunks per workgroup (never across a segment)
    const long long nblk = (long long)a.B * a.H * ((nc + 1) / 2);
    hipLaunchKernelGGL((clean_out_kernel<T, DK, 2>), dim3((unsigned)nblk), dim3(2 * kThreads), 0, st, a);
  } else {
    const long long nblk = (long long)a.B * a.H * nc;
    hipLaunchKernelGGL((clean_out_kernel<T, DK, 1>), dim3((unsigned)nblk), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

#define CCQ_CLEAN_DISPATCH(fn, a, bf, st)                      \
  do {                                                         \
    if (bf) {                                                  \
      switch ((a).dk) {                                        \
        case 64: return fn<bf16_t, 64>((a), (st));             \
        case 128: return fn<bf16_t, 128>((a), (st));           \
        case 256: return fn<bf16_t, 256>((a), (st));           \
      }                                                        \
    } else {                                                   \
      switch ((a).dk) {                                        \
        case 64: return fn<float, 64>((a), (st));              \
        case 128: return fn<float, 128>((a), (st));            \
      }                                                        \
    }                                                          \
    return hipErrorInvalidValue;                               \
  } while (0)
}  // namespace

bool clean_supported(int dk, bool is_bf16) {
  if (is_bf16) return dk == 64 || dk == 128 || dk == 256;
  return dk == 64 || dk == 128;
}

hipError_t launch_clean_gram(const CleanArgs& a, bool is_bf16, hipStream_t st) {
  CCQ_CLEAN_DISPATCH(run_gram, a, is_bf16, st);
}

hipError_t launch_clean_prefix(const CleanArgs& a, bool is_bf16, hipStream_t st) {
  CCQ_CLEAN_DISPATCH(run_prefix, a, is_bf16, st);
}

hipError_t launch_clean_out(const CleanArgs& a, bool is_bf16, hipStream_t st) {
  CCQ_CLEAN_DISPATCH(run_out, a, is_bf16, st);
}

}  // namespace ccq
