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
//   clean_out     one workgroup per segment: walks its chunks in order with
//                 S'_r (S'_s plus the centred keys of the segment's earlier
//                 chunks) held in MFMA accumulators
// Without centring (Sigma = Cbar) the same kernels run with c_s = 0 and no
// mean terms.
//
// Decay-aligned statistics (DECAY; Gated DeltaNet's scalar decay alpha_t):
// key j enters token t's sums with weight w_{j,t} = e^{L_t - L_j} (L the
// cumulative log decay) and t becomes W_t = sum_{j<=t} w_{j,t}.  Every sum
// is kept decayed to the point it is taken at: the Gram and key sums of a
// chunk or segment to its end, the carried moment of clean_out to the chunk
// it enters; a sum moves on by one chunk as  X <- e^{gamma_C} X + (the chunk's
// terms weighted e^{gamma_C - gamma_j})  (gamma the chunk's inclusive log-decay
// prefix), and within a chunk token i sees e^{gamma_i} times the chunk-entry
// sums plus its keys weighted e^{gamma_i - gamma_j}.  The shift invariance
// above holds for the weighted covariance too (with W in place of t), so the
// segment centring is unchanged; c_s is the segment's weighted mean.  Every
// factor is at most 1.
#include <type_traits>

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
// from the same products (a ones column).
// DECAY: each chunk's rows are staged times sqrt(e^{gamma_C - gamma_j}) (so the
// product of two of them carries the weight once), the ones column becomes
// the column of those square roots, and the sums so far are decayed by the
// chunk's e^{gamma_C} before its terms are added; also each segment's weight
// sum and decay (sdec).
template <typename T, int DK, bool DECAY>
__global__ __launch_bounds__(64 * (DK >= 128 ? 8 : 4), 1) void clean_gram_kernel(const CleanArgs a) {
  constexpr int C = kChunk, P = Pad<T>::value, LDK = DK + P;
  constexpr int NWG = DK >= 128 ? 8 : 4, NTG = 64 * NWG;
  constexpr int RW = DK / NWG;  // rows per wave
  constexpr int RT = RW / 16;   // row tiles per wave
  constexpr int CT = DK / 16;   // column tiles
  __shared__ __align__(16) T sK[2][C * LDK];
  // DECAY, per chunk parity: sqrt of each row's weight, and the chunk's decay
  __shared__ __align__(16) float sW[2][DECAY ? C : 1];
  __shared__ float sDc[2];

  const int NC = n_chunks(a.T), NS = n_segs(a.T, a.seg);
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / NS, s = lb % NS;
  const int b = bh / a.H, h = bh % a.H;
  const int w = wave_id(), l = lane_id(), g4 = l >> 4, c16 = l & 15;
  const int a0 = w * RW;
  const T* k = static_cast<const T*>(a.k);
  const size_t gstride = (size_t)a.H * DK;
  const Seq sq = seq_of(a.cu, b, a.T);
  // a packed sequence's segments past its end are empty: zero sums
  const int cbeg = s * a.seg, cend = min(n_chunks(sq.len), cbeg + a.seg);

  f32x4 acc[RT][CT], stot[RT];
#pragma unroll
  for (int v = 0; v < RT; ++v) {
    stot[v] = zero4();
#pragma unroll
    for (int t = 0; t < CT; ++t) acc[v][t] = zero4();
  }

  RowTile<T, DK, NTG> rk;
  RowScales<RowTile<T, DK, NTG>> fk;
  float lav = 0.f;    // DECAY, wave 0: the log decay of row l of the next chunk
  float om = 0.f;     // DECAY, wave 0: the segment's weight sum so far
  float lseg = 0.f;   // DECAY, wave 0: the segment's log decay so far
  auto load = [&](int c) {
    const int n = min(C, sq.len - c * C);
    rk.load(k + seq_off(sq, c * C, h, a.H, DK), gstride, n);
    if (a.rk) fk.load(a.rk + seq_idx(sq, c * C, h, a.H), (size_t)a.H, n);
    if constexpr (DECAY)
      if (w == 0) lav = l < n ? a.la[seq_idx(sq, c * C + l, h, a.H)] : 0.f;
  };
  if (cbeg < cend) load(cbeg);
  const Frag<T> ones = ones_col_frag<T>();

  for (int c = cbeg; c < cend; ++c) {
    const int par = (c - cbeg) & 1;
    T* buf = sK[par];  // the other buffer may still be read by a slower wave
    if constexpr (DECAY) {
      if (w == 0) {
        // inclusive log-decay prefix over the chunk's rows (lane = row)
        float g = lav;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const float u = __shfl_up(g, o);
          if (l >= o) g += u;
        }
        const float gC = __shfl(g, 63);  // rows past the end add nothing
        const int n = min(C, sq.len - c * C);
        const float wj = l < n ? __expf(gC - g) : 0.f;
        sW[par][l] = l < n ? __expf(0.5f * (gC - g)) : 0.f;
        float ws = wj;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) ws += __shfl_xor(ws, o);
        om = __expf(gC) * om + ws;
        lseg += gC;
        if (l == 0) sDc[par] = __expf(gC);
      }
      lds_barrier();  // the chunk's weights
#pragma unroll
      for (int u = 0; u < RowTile<T, DK, NTG>::NV; ++u)
        if (RowTile<T, DK, NTG>::mine(u)) {
          const float f = sW[par][RowTile<T, DK, NTG>::row(u)] * (a.rk ? fk.f[u] : 1.f);
#pragma unroll
          for (int e = 0; e < 8; ++e) rk.v[u][e] = to<T>(f32(rk.v[u][e]) * f);
        }
    } else {
      if (a.rk) fk.apply(rk);
    }
    rk.store(buf, LDK);
    if (c + 1 < cend) load(c + 1);
    lds_barrier();  // (LDS only: a __syncthreads() fence would wait for the load just issued)
    if constexpr (DECAY) {  // the sums so far, decayed to this chunk's end
      const float dc = sDc[par];
#pragma unroll
      for (int v = 0; v < RT; ++v) {
        stot[v] *= dc;
#pragma unroll
        for (int t = 0; t < CT; ++t) acc[v][t] *= dc;
      }
    }
    f32x4 msum[RT];
#pragma unroll
    for (int v = 0; v < RT; ++v) msum[v] = zero4();
#pragma unroll
    for (int k0 = 0; k0 < C; k0 += 32) {
      Frag<T> col = ones;  // DECAY: column 0 holds the square roots of the rows' weights
      if constexpr (DECAY) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          set_frag_elem(col, e, c16 == 0 ? sW[par][k0 + 8 * g4 + e] : 0.f);
      }
      Frag<T> fa[RT];
#pragma unroll
      for (int v = 0; v < RT; ++v) {
        fa[v] = ld_frag_tr(buf + k0 * LDK + a0 + 16 * v, LDK);
        mma(msum[v], fa[v], col);
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
  if constexpr (DECAY)
    if (w == 0 && l == 0) {  // (an empty segment: no weight, no decay)
      a.sdec[((size_t)bh * NS + s) * 2] = om;
      a.sdec[((size_t)bh * NS + s) * 2 + 1] = __expf(lseg);
    }
  // acc[v][t] is accumulator tile (rows m = a0 + 16 v .., columns n = 16 t ..),
  // stored fragment-native: 1 KB per tile, lane-contiguous
  float* G = a.gram + ((size_t)bh * NS + s) * DK * DK;
#pragma unroll
  for (int v = 0; v < RT; ++v)
#pragma unroll
    for (int t = 0; t < CT; ++t)
      *reinterpret_cast<f32x4*>(G + ((size_t)(t * CT + a0 / 16 + v) * 64 + l) * 4) = acc[v][t];
}

// S'_s = S_s - M'_s c_s^T - c_s M'_s^T - n_s c_s c_s^T with S_s the raw second
// moment before segment s (prefix of the Gram matrices, fp32), c_s the mean
// key of segment s, n_s the tokens before it and M'_s = M_s - n_s c_s the key
// sum before it about c_s (running sums of the segment key sums).  Each thread
// owns four consecutive fragment-native elements, (m .. m + 3, n): one scalar
// index n and a vector of four m.  Also the final Cbar_T and mu_T.
// DECAY: the prefix runs over the segments decayed, X <- E_s X + (segment s's
// sum, decayed to its end), and the segment's and the earlier tokens' decayed
// weight sums take the place of the token counts (t0 = 0, no C0 / mu0).
template <typename T, int DK, bool DECAY>
__global__ __launch_bounds__(256) void clean_prefix_kernel(const CleanArgs a) {
  constexpr int PER = DK * DK / 4 / 256;  // workgroups per head
  constexpr int NMT = DK / 16;
  const int bh = blockIdx.x / PER;
  const int g = (blockIdx.x % PER) * 256 + threadIdx.x;  // element offset / 4
  const int l = g & 63, tile = g >> 6;
  const int n = 16 * (tile / NMT) + (l & 15);
  const int m = 16 * (tile % NMT) + 4 * (l >> 4);
  const int NS = n_segs(a.T, a.seg);
  const Seq sq = seq_of(a.cu, bh / a.H, a.T);
  const int NSL = n_segs(sq.len, a.seg), NCL = n_chunks(sq.len);  // this sequence's own
  const float t0f = (float)a.t0;
  f32x4 acc = zero4();
  if (a.C0) acc = *reinterpret_cast<const f32x4*>(a.C0 + ((size_t)bh * DK + n) * DK + m) * t0f;
  float run_a = a.mu0 ? t0f * a.mu0[(size_t)bh * DK + n] : 0.f;  // raw key sums before s
  f32x4 run_b = a.mu0 ? *reinterpret_cast<const f32x4*>(a.mu0 + (size_t)bh * DK + m) * t0f : zero4();
  T* Sp = static_cast<T*>(a.sprime);
  float wb = 0.f;  // DECAY: decayed weight of the tokens before segment s
  for (int s = 0; s < NSL; ++s) {
    const size_t so = (size_t)bh * NS + s;
    const int cbeg = s * a.seg, cend = min(NCL, cbeg + a.seg);
    float len = (float)(min(sq.len, cend * kChunk) - cbeg * kChunk);
    float ns = t0f + (float)((int64_t)cbeg * kChunk);
    float E = 1.f;
    if constexpr (DECAY) {
      len = a.sdec[so * 2];
      E = a.sdec[so * 2 + 1];
      ns = wb;
    }
    const float tot_a = a.ssum[so * DK + n];
    const f32x4 tot_b = *reinterpret_cast<const f32x4*>(a.ssum + so * DK + m);
    const f32x4 gm = *reinterpret_cast<const f32x4*>(a.gram + so * DK * DK + 4 * (size_t)g);
    const float ca = a.centered ? tot_a / len : 0.f;
    const f32x4 cb4 = a.centered ? tot_b / len : zero4();
    const float ma = run_a - ns * ca;
    const f32x4 mb4 = run_b - ns * cb4;
    f32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = acc[q] - ma * cb4[q] - ca * mb4[q] - ns * ca * cb4[q];
    store4(Sp + so * DK * DK + 4 * (size_t)g, o[0], o[1], o[2], o[3]);
    if constexpr (DECAY) {
      acc = acc * E + gm;
      run_a = run_a * E + tot_a;
      run_b = run_b * E + tot_b;
      wb = wb * E + len;
    } else {
      acc += gm;
      run_a += tot_a;
      run_b += tot_b;
    }
  }
  if (a.t0 + sq.len == 0) {  // no token at all (an empty packed sequence): the initial cache
    if (a.CT)
      *reinterpret_cast<f32x4*>(a.CT + ((size_t)bh * DK + n) * DK + m) =
          a.C0 ? *reinterpret_cast<const f32x4*>(a.C0 + ((size_t)bh * DK + n) * DK + m) : zero4();
    if (a.muT && n == 0)
      *reinterpret_cast<f32x4*>(a.muT + (size_t)bh * DK + m) =
          a.mu0 ? *reinterpret_cast<const f32x4*>(a.mu0 + (size_t)bh * DK + m) : zero4();
    return;
  }
  const float inv = 1.f / (DECAY ? wb : t0f + (float)sq.len);  // W_T for the decayed sums
  if (a.CT) *reinterpret_cast<f32x4*>(a.CT + ((size_t)bh * DK + n) * DK + m) = acc * inv;
  if (a.muT && n == 0) *reinterpret_cast<f32x4*>(a.muT + (size_t)bh * DK + m) = run_b * inv;
}

// Transposed fragment at a lane-offset pointer (frag_tr_at); for bf16 the two
// reads are issued as inline assembly so that the compiler does not drain the
// streamed prefetch before them (the caller waits with lds_wait).
template <typename T>
__device__ __forceinline__ Frag<T> frag_tr_any(const T* p, int ld) {
  if constexpr (sizeof(T) == 2) {
    const bf16x4 lo = ds_read_tr16_asm(p), hi = ds_read_tr16_asm(p + 4 * ld);
    Frag<T> f;
    f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return f;
  } else {
    return frag_tr_at(p, ld);
  }
}

// Causal score tile t of a 64-token chunk (t < 10): key tile J <= token tile I.
__device__ __forceinline__ int causal_tile_i(int t) { return t >= 6 ? 3 : t >= 3 ? 2 : t >= 1 ? 1 : 0; }

// One workgroup per (head, segment) walks the segment's chunks in order with
// S'_r, the second moment about c_s of every key before chunk r, held in MFMA
// accumulators: wave w owns columns n in [w NCW, (w + 1) NCW) of S' and all
// of its rows.  Per chunk r (x: the chunk's rows of q, K': its keys minus c_s):
//   out^T  = S'_r x^T                  (S' enters as bf16 operands from registers)
//   sc     = K' x^T, masked to j <= i and shifted by -cq'_i / t_i
//   out^T += K'^T sc
//   S'_{r+1} = S'_r + K'^T K'
// The shift folds the within-chunk part of the mean term into the product;
// cq'_i = m'_i . x_i comes from the score row sums and M'_r . x_i.  x and K'
// are staged in LDS once per chunk; q_clean is formed in place over x and is
// copied out with row-contiguous stores while the next chunk is staged.
// DECAY (the decay-aligned statistics): with gamma the chunk's inclusive
// log-decay prefix and W_i token i's decayed count,
//   out^T  = diag(e^{gamma_i}) S'_r x^T + K'^T sc,   sc_ij scaled e^{gamma_i - gamma_j}
//   cq'_i  = e^{gamma_i} M'_r . x_i + sum_{j <= i} sc_ij,  shift cq'_i / W_i (times
//            the weight), mean term e^{gamma_i} (cq'_i / W_i) M'_r, all over W_i
//   S'_{r+1} = e^{gamma_C} S'_r + K'^T diag(e^{gamma_C - gamma}) K',
//   M'_{r+1} = e^{gamma_C} M'_r + (the chunk's weighted key sum about c_s).
template <typename T, int DK, int NW, bool TRAIN, bool DECAY>
__global__ __launch_bounds__(64 * NW, 1) void clean_out_kernel(const CleanArgs a) {
  // the shifted scores overwrite the raw ones in place (row i of both is
  // written and read only by the threads of token i, one wave, whose LDS
  // accesses complete in order), which leaves room at dk = 256 for the 32-byte
  // row padding; a row of raw scores is 288 bytes, so the shifted scores'
  // fragment reads see the same conflict-free 32 mod 256 pitch
  constexpr int C = kChunk, P = Pad<T>::value, LDK = DK + P, LDQ = C + 8;
  constexpr int LDP = LDQ * 4 / (int)sizeof(T);
  constexpr int NT = 64 * NW, VPR = DK / 8;
  constexpr int NCW = DK / NW, NNT = NCW / 16, NMT = DK / 16, NK = DK / 32;
  constexpr int TPI = NT / C, JPT = C / TPI, FPT = DK / TPI;  // per-token split of the row sums
  constexpr int NV = C * VPR / NT;                            // staged vectors per thread
  static_assert(NCW % 16 == 0 && NNT >= 1, "column split");
  static_assert(NT >= DK && JPT % 8 == 0 && FPT % 8 == 0 && C * VPR % NT == 0 && NT % VPR == 0, "thread split");
  typedef RowTile<T, DK, NT> Tile;
  typedef typename Tile::vec_t vec_t;
  // bf16 chunks are prefetched straight into LDS (x then k, unpadded); fp32
  // ones, whose staging area would not fit beside the rest, into registers.
  // One LDS block, hot arrays first so that their offsets fit in the
  // instructions' immediate field.
  constexpr bool kDma = sizeof(T) == 2;
  constexpr int oX = 0, oK = oX + C * LDK * (int)sizeof(T), oS = oK + C * LDK * (int)sizeof(T);
  constexpr int oC = oS + C * LDQ * 4, oM = oC + DK * 4;
  constexpr int oCq = oM + DK * 4, oLam = oCq + C * 4, oDec = oLam + C * 4;
  constexpr int oSt = oDec + (DECAY ? (3 * C + 4) * 4 : 0);
  constexpr int oEnd = oSt + (kDma ? 2 * C * DK * (int)sizeof(T) : 16);
  __shared__ __align__(16) char smem[oEnd];
  T* const sX = reinterpret_cast<T*>(smem + oX);         // x rows, then q_clean rows
  T* const sK = reinterpret_cast<T*>(smem + oK);         // centred keys
  float* const sS = reinterpret_cast<float*>(smem + oS); // raw scores, [i][j]
  T* const sP = reinterpret_cast<T*>(smem + oS);         // masked, shifted scores, [i][j], over sS
  float* const sC = reinterpret_cast<float*>(smem + oC);
  float* const sM = reinterpret_cast<float*>(smem + oM);
  float* const sCq = reinterpret_cast<float*>(smem + oCq);
  float* const sLam = reinterpret_cast<float*>(smem + oLam);
  T* const sSt = reinterpret_cast<T*>(smem + oSt);
  // DECAY: gamma_i, e^{gamma_i}, W_i of the chunk's tokens, and [0] W entering the
  // chunk, [1] e^{gamma_C} and [2] the weight sum of the previous chunk, [3] W
  // leaving this chunk
  float* const sGm = reinterpret_cast<float*>(smem + oDec);
  float* const sEg = sGm + C;
  float* const sWt = sGm + 2 * C;
  float* const sSc = sGm + 3 * C;
  static_assert(!(DECAY && sizeof(T) == 2 && DK == 256 && oEnd > 160 * 1024), "LDS");

  const int NC = n_chunks(a.T), NS = n_segs(a.T, a.seg);
  const int lb = xcd_logical_block(blockIdx.x, gridDim.x);
  const int bh = lb / NS, s = lb % NS;
  const int b = bh / a.H, h = bh % a.H;
  const Seq sq = seq_of(a.cu, b, a.T);
  // rows of the token tensors this kernel writes (q_clean and, in training,
  // Sigma x, m . x and the base), which live in the workspace in a padded
  // [B, T, ...] layout whatever the layout of the inputs
  const Seq sw{(long long)b * a.T, sq.len};
  const int cbeg = s * a.seg, cend = min(n_chunks(sq.len), cbeg + a.seg);
  if (cbeg >= cend) return;  // a segment past a packed sequence's end
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = w * NCW;
  const T* x = static_cast<const T*>(a.q);
  const T* k = static_cast<const T*>(a.k);
  T* qc = static_cast<T*>(a.qclean);
  const size_t gstride = (size_t)a.H * DK;
  const float t0f = (float)a.t0;
  const size_t so = (size_t)bh * NS + s;

  Tile rx, rk;
  RowScalar rl, rla;  // lambda and (DECAY) the log decay of token tid
  // row scales of raw q and k (l2 normalisation folded in), for the rows of
  // this thread's staged vectors
  float fq[NV], fk[NV];
  // streamed chunk: piece i of the x rows for i < NI, of the key rows after
  typedef LdsStream<DK, NW> Stream;
  auto stream_piece = [&](int c, int i) {
    if constexpr (kDma) {
      const int r0 = c * C, n = min(C, sq.len - r0);
      if (i < Stream::NI) Stream::load_one(x + seq_off(sq, r0, h, a.H, DK), gstride, n, sSt, i);
      else Stream::load_one(k + seq_off(sq, r0, h, a.H, DK), gstride, n, sSt + C * DK, i - Stream::NI);
    }
  };
  // everything but the streamed pieces when `spread` (those then go out one
  // or two at a time between the next products)
  auto prefetch = [&](int c, bool spread) {
    const int r0 = c * C, n = min(C, sq.len - r0);
    if (a.rq) {
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int row = min((tid + NT * u) / VPR, n - 1);
        fq[u] = a.rq[seq_idx(sq, r0 + row, h, a.H)];
        fk[u] = a.rk[seq_idx(sq, r0 + row, h, a.H)];
      }
    }
    if constexpr (kDma) {
      if (!spread)
#pragma unroll
        for (int i = 0; i < 2 * Stream::NI; ++i) stream_piece(c, i);
    } else {
      rx.load(x + seq_off(sq, r0, h, a.H, DK), gstride, n);
      rk.load(k + seq_off(sq, r0, h, a.H, DK), gstride, n);
    }
    if (tid < C) rl.load(a.lam + seq_idx(sq, r0, h, a.H), (size_t)a.H, tid, n);
    if (DECAY && tid < C) rla.load(a.la + seq_idx(sq, r0, h, a.H), (size_t)a.H, tid, n);
  };
  prefetch(cbeg, false);

  // segment centre c_s and key sum before the segment about it, M'_s; one
  // thread per feature
  float cen = 0.f;
  if (tid < DK) {
    const float* ss = a.ssum + (size_t)bh * NS * DK + tid;
    if constexpr (DECAY) {
      // decayed key sum and weight before the segment (segment sums decayed
      // to their ends, carried through the later segments' decays)
      const float* sd = a.sdec + (size_t)bh * NS * 2;
      float run = 0.f, wb = 0.f;
      for (int p = 0; p < s; ++p) {
        run = run * sd[2 * p + 1] + ss[(size_t)p * DK];
        wb = wb * sd[2 * p + 1] + sd[2 * p];
      }
      cen = a.centered ? ss[(size_t)s * DK] / sd[2 * s] : 0.f;
      sC[tid] = cen;
      sM[tid] = run - wb * cen;
      if (tid == 0) sSc[3] = wb;  // W entering the segment's first chunk
    } else {
      float run = a.mu0 ? t0f * a.mu0[(size_t)bh * DK + tid] : 0.f;
#pragma unroll 8
      for (int p = 0; p < s; ++p) run += ss[(size_t)p * DK];
      const float len = (float)(min(sq.len, cend * C) - cbeg * C);
      cen = a.centered ? ss[(size_t)s * DK] / len : 0.f;
      sC[tid] = cen;
      sM[tid] = run - (t0f + (float)((int64_t)cbeg * C)) * cen;
    }
  }
  // entry moment S'_s, held with its rows in pair order: accumulator row
  // 4 g + r of tile mt is feature pair_feat(mt, g, r) = 32 (mt / 2) + 8 g +
  // 4 (mt % 2) + r, so that two tiles pack into an operand fragment whose k
  // slots are 8 consecutive features (one 16-byte LDS read for the matching
  // x fragment).  The stored layout is fragment-native in natural row order
  // (rows m = 16 mt + 4 (l / 16) + r, column n0 + 16 nt + l % 16): tile mt,
  // lane group g reads its 4 rows from tile 2 (mt / 2) + g / 2, group
  // 2 (g % 2) + mt % 2.
  f32x4 S[NNT][NMT];
  {
    const int lg = (tid & 63) >> 4, lc = tid & 15;
    const T* sp = static_cast<const T*>(a.sprime) + so * DK * DK + (size_t)(n0 / 16) * NMT * 64 * 4;
#pragma unroll
    for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) {
        const int mo = 2 * (mt >> 1) + (lg >> 1), go = 2 * (lg & 1) + (mt & 1);
        S[nt][mt] = load4f(sp + (((size_t)nt * NMT + mo) * 64 + 16 * go + lc) * 4);
      }
  }
  if constexpr (kDma) wait_vm_all();
  __syncthreads();  // sC, first chunk

  float csum = 0.f;  // key sum of the current chunk, feature tid
  for (int c = cbeg; c < cend; ++c) {
    const int r0 = c * C, nrow = min(C, sq.len - r0);
    // per-token and per-feature values first: waiting for their loads costs
    // nothing here, while after the stores below it would also wait for those
    if (tid < C) sLam[tid] = rl.get();
    if constexpr (DECAY) {
      if (tid < 64) {  // wave 0: the chunk's inclusive log-decay prefix (lane = token)
        float g = rla.get();
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const float u = __shfl_up(g, o);
          if (tid >= o) g += u;
        }
        sGm[tid] = g;
        sEg[tid] = __expf(g);
      }
      if (tid == 0) sSc[0] = sSc[3];  // W entering this chunk
    }
    if (tid < DK) {
      if (c > cbeg) {  // M'_c
        if constexpr (DECAY) sM[tid] = sSc[1] * sM[tid] + (csum - sSc[2] * cen);
        else sM[tid] += csum - (float)C * cen;
      }
      csum = a.csum[((size_t)bh * NC + c) * DK + tid];
    }
    // stage chunk c; each thread first copies out the q_clean of chunk c - 1
    // (always a full chunk) held at the same places.  The outgoing rows and the
    // centre are read together and stored before the streamed chunk is read
    // (two LDS round trips per chunk, few registers); a register-prefetched
    // chunk is taken first instead, so that its wait covers no store.
    {
      const int t_ = opaque(tid);
      const int col = (t_ % VPR) * 8;  // the same for every vector of a thread
      vec_t xv[NV], kv[NV];
      auto take = [&]() {
#pragma unroll
        for (int u = 0; u < NV; ++u) {
          if constexpr (kDma) {
            xv[u] = *reinterpret_cast<const vec_t*>(sSt + 8 * (t_ + NT * u));
            kv[u] = *reinterpret_cast<const vec_t*>(sSt + C * DK + 8 * (t_ + NT * u));
          } else {
            xv[u] = rx.get(u);
            kv[u] = rk.get(u);
          }
        }
        if (a.rq)
#pragma unroll
          for (int u = 0; u < NV; ++u)
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              xv[u][q] = to<T>(f32(xv[u][q]) * fq[u]);
              kv[u][q] = to<T>(f32(kv[u][q]) * fk[u]);
            }
      };
      if constexpr (!kDma) take();
      const f32x4 ca = *reinterpret_cast<const f32x4*>(sC + col);
      const f32x4 cb = *reinterpret_cast<const f32x4*>(sC + col + 4);
      if (c > cbeg) {
        vec_t qo[NV];
#pragma unroll
        for (int u = 0; u < NV; ++u) qo[u] = *reinterpret_cast<const vec_t*>(sX + ((t_ + NT * u) / VPR) * LDK + col);
#pragma unroll
        for (int u = 0; u < NV; ++u)
          *reinterpret_cast<vec_t*>(qc + seq_off(sw, r0 - C + (t_ + NT * u) / VPR, h, a.H, DK) + col) = qo[u];
      }
      if constexpr (kDma) take();
      auto put = [&](auto masked) {
#pragma unroll
        for (int u = 0; u < NV; ++u) {
          const int row = (t_ + NT * u) / VPR;
          const bool live = row < nrow;
          const float keep = live ? 1.f : 0.f;  // (a product, not a select: no branch per element)
          vec_t y;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float d = f32(kv[u][q]) - (q < 4 ? ca[q] : cb[q - 4]);
            if constexpr (decltype(masked)::value) {
              xv[u][q] = live ? xv[u][q] : to<T>(0.f);
              y[q] = to<T>(d * keep);
            } else {
              y[q] = to<T>(d);
            }
          }
          *reinterpret_cast<vec_t*>(sX + row * LDK + col) = xv[u];
          *reinterpret_cast<vec_t*>(sK + row * LDK + col) = y;
        }
      };
      // rows past the end exist only in a sequence's last chunk
      if (nrow == C) put(std::false_type{});
      else put(std::true_type{});
    }
    lds_barrier();  // (1) x, K', M'_c staged; the staging area is free
    const bool more = c + 1 < cend;
    if (more) prefetch(c + 1, true);

    // raw scores of the causal tiles this wave owns, to sS[i][j]; then
    // out^T = S'_r x^T: acc[nt][I] holds features n0 + 16 nt + 4 (l / 16) + r
    // of token 16 I + l % 16
    f32x4 acc[NNT][4];
    {
      const int l_ = opaque(tid & 63), g_ = l_ >> 4, c_ = l_ & 15;
      // x fragments in natural feature order: one 16-byte read per lane
      const T* px8 = sX + c_ * LDK + 8 * g_;
      {
        const T* pk8 = sK + c_ * LDK + 8 * g_;
        for (int t = w; t < 10; t += NW) {
          const int I = causal_tile_i(t), J = t - I * (I + 1) / 2;
          f32x4 sc = zero4();
#pragma unroll
          for (int p = 0; p < NK; ++p) mma(sc, frag_at(pk8 + 16 * J * LDK + 32 * p), frag_at(px8 + 16 * I * LDK + 32 * p));
          *reinterpret_cast<f32x4*>(sS + (16 * I + c_) * LDQ + 16 * J + 4 * g_) = sc;
        }
      }
#pragma unroll
      for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
        for (int I = 0; I < 4; ++I) acc[nt][I] = zero4();
#pragma unroll
      for (int p = 0; p < NK; ++p) {
        Frag<T> xf[4], af[NNT];
#pragma unroll
        for (int I = 0; I < 4; ++I) xf[I] = frag_at(px8 + 16 * I * LDK + 32 * p);
#pragma unroll
        for (int nt = 0; nt < NNT; ++nt) af[nt] = acc_pair_frag<T>(S[nt][2 * p], S[nt][2 * p + 1]);
#pragma unroll
        for (int I = 0; I < 4; ++I)
#pragma unroll
          for (int nt = 0; nt < NNT; ++nt) mma(acc[nt][I], af[nt], xf[I]);
        // the next chunk's streamed pieces, spread over these products
        if constexpr (kDma) {
          constexpr int PPS = (2 * Stream::NI + NK - 1) / NK;
#pragma unroll
          for (int i = PPS * p; i < PPS * (p + 1); ++i)
            if (i < 2 * Stream::NI && more) stream_piece(c + 1, i);
        }
      }
    }
    lds_barrier();  // (2) scores complete

    // cq'_i = M'_r . x_i + sum_{j <= i} sc_ij, and the shifted scores; TPI
    // consecutive threads per token
    {
      const int t_ = opaque(tid);
      const int i = t_ / TPI, pp = t_ % TPI;
      float ti = t0f + (float)(r0 + i + 1);  // DECAY: becomes W_i below
      float sv[JPT];
      float rs = 0.f, mq = 0.f, cx = 0.f, ws = 0.f;
      const float* srow = sS + i * LDQ + JPT * pp;
#pragma unroll
      for (int e = 0; e < JPT; e += 4) {
        const f32x4 v4 = *reinterpret_cast<const f32x4*>(srow + e);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = JPT * pp + e + q;
          if constexpr (DECAY) {  // weight e^{gamma_i - gamma_j} (0 past the diagonal)
            const float f = j <= i ? __expf(sGm[i] - sGm[j]) : 0.f;
            ws += f;
            sv[e + q] = f * v4[q];
          } else {
            sv[e + q] = j <= i ? v4[q] : 0.f;
          }
          rs += sv[e + q];
        }
      }
      // this thread's features are the 4-wide groups pp, pp + TPI, ...: the TPI
      // threads of a token read adjacent 8- and 16-byte pieces (no bank conflicts)
      const T* xrow = sX + i * LDK + 4 * pp;
      const float* mrow = sM + 4 * pp;
      const float* crow = sC + 4 * pp;
#pragma unroll
      for (int e = 0; e < FPT; e += 4) {
        const int f = TPI * e;  // = 4 TPI (e / 4)
        float xv[4];
        if constexpr (sizeof(T) == 2) {
          const bf16x4 x4 = *reinterpret_cast<const bf16x4*>(xrow + f);
#pragma unroll
          for (int q = 0; q < 4; ++q) xv[q] = f32(x4[q]);
        } else {
          const f32x4 x4 = *reinterpret_cast<const f32x4*>(xrow + f);
#pragma unroll
          for (int q = 0; q < 4; ++q) xv[q] = x4[q];
        }
        const f32x4 m4 = *reinterpret_cast<const f32x4*>(mrow + f);
        const f32x4 c4 = *reinterpret_cast<const f32x4*>(crow + f);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          mq += xv[q] * m4[q];
          cx += xv[q] * c4[q];
        }
      }
      rs = group_sum<TPI>(rs);
      mq = group_sum<TPI>(mq);
      cx = group_sum<TPI>(cx);
      if constexpr (DECAY) {
        const float eg = sEg[i];
        mq *= eg;                               // the chunk-entry sum decayed to token i
        ti = eg * sSc[0] + group_sum<TPI>(ws);  // W_i
      }
      const float cqp = mq + rs;
      const float sub = a.centered ? cqp / ti : 0.f;
      // the shifted row goes over the raw one: keep these stores after the reads
      asm volatile("" ::: "memory");
      T* prow = sP + i * LDP + JPT * pp;
#pragma unroll
      for (int e = 0; e < JPT; e += 8) {
        vec_t y;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if constexpr (DECAY) {  // the weight again (zero past the diagonal)
            const int j = JPT * pp + e + q;
            y[q] = to<T>(j <= i ? sv[e + q] - __expf(sGm[i] - sGm[j]) * sub : 0.f);
          }
          else y[q] = to<T>(JPT * pp + e + q <= i ? sv[e + q] - sub : 0.f);
        }
        *reinterpret_cast<vec_t*>(prow + e) = y;
      }
      if (pp == 0) {
        sCq[i] = cqp;
        if constexpr (DECAY) {
          sWt[i] = ti;
          if (i == C - 1) {  // W leaving the chunk, its decay and its own weight sum
            sSc[3] = ti;
            sSc[1] = sEg[C - 1];
            sSc[2] = ti - sEg[C - 1] * sSc[0];
          }
        }
        if (TRAIN && a.mdot && i < nrow) a.mdot[seq_idx(sw, r0 + i, h, a.H)] = cqp + ti * cx;  // raw m . x
      }
    }
    lds_barrier();  // (3) shifted scores complete

    {
      const int l_ = opaque(tid & 63), g_ = l_ >> 4, c_ = l_ & 15;
      const T* ptr = sK + frag_tr_lane_off<T>(l_, LDK);
      // K'^T rows in the pair order of the moment's tiles (the update)
      const T* ptr_pair = sK + frag_tr_pair_lane_off<T>(l_, LDK);
      // K'^T fragments of this wave's columns (intra-chunk product and update)
      Frag<T> kb[NNT][2];
#pragma unroll
      for (int nt = 0; nt < NNT; ++nt)
#pragma unroll
        for (int q = 0; q < 2; ++q) kb[nt][q] = frag_tr_any(ptr + 32 * q * LDK + n0 + 16 * nt, LDK);
      if constexpr (kDma)
#pragma unroll
        for (int nt = 0; nt < NNT; ++nt) lds_wait(kb[nt]);
      if constexpr (DECAY)  // the chunk-entry moment's part, decayed to each token
#pragma unroll
        for (int I = 0; I < 4; ++I) {
          const float eg = sEg[16 * I + c_];
#pragma unroll
          for (int nt = 0; nt < NNT; ++nt) acc[nt][I] *= eg;
        }
      // out^T += K'^T sc (keys 32..63 only reach tokens 32..63)
      const T* pp_ = sP + c_ * LDP + 8 * g_;
#pragma unroll
      for (int I = 0; I < 4; ++I)
#pragma unroll
        for (int q = 0; q < (I >= 2 ? 2 : 1); ++q) {
          const Frag<T> pf = frag_at(pp_ + 16 * I * LDP + 32 * q);
#pragma unroll
          for (int nt = 0; nt < NNT; ++nt) mma(acc[nt][I], kb[nt][q], pf);
        }

      // q_clean = base - lam / t (out - cq' / t M'_r), written over x
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        const int i = 16 * I + c_;
        f32x4 xb[NNT];
#pragma unroll
        for (int nt = 0; nt < NNT; ++nt) {
          const int n = n0 + 16 * nt + 4 * g_;
          if constexpr (TRAIN)
            xb[nt] = a.base ? *reinterpret_cast<const f32x4*>(a.base + seq_off(sw, r0 + min(i, nrow - 1), h, a.H, DK) + n)
                            : load4f(sX + i * LDK + n);
          else
            xb[nt] = load4f(sX + i * LDK + n);
        }
        const float inv = 1.f / (DECAY ? sWt[i] : t0f + (float)(r0 + i + 1));
        const float msub = a.centered ? (DECAY ? sEg[i] : 1.f) * sCq[i] * inv : 0.f;
        const float lam = sLam[i], li = lam * inv, lm = li * msub;
#pragma unroll
        for (int nt = 0; nt < NNT; ++nt) {
          const int n = n0 + 16 * nt + 4 * g_;
          const f32x4 mr = *reinterpret_cast<const f32x4*>(sM + n);
          // o = base - (lam / t) out + (lam / t) msub M'_r, two products per element
          f32x4 cr, o;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            o[r] = fmaf(-li, acc[nt][I][r], fmaf(lm, mr[r], xb[nt][r]));
            if constexpr (TRAIN) cr[r] = (acc[nt][I][r] - msub * mr[r]) * inv;  // Sigma_t x_t
          }
          store4(sX + i * LDK + n, o[0], o[1], o[2], o[3]);
          if (TRAIN && i < nrow) {
            const size_t off = seq_off(sw, r0 + i, h, a.H, DK) + n;
            if (a.qclean_dbg) *reinterpret_cast<f32x4*>(a.qclean_dbg + off) = o;
            if (a.corr) *reinterpret_cast<f32x4*>(a.corr + off) = cr;
          }
        }
      }

      // S'_{r+1} = S'_r + K'^T K' (not needed after the segment's last chunk);
      // transposed key reads two m tiles ahead of their products
      if (c + 1 < cend) {
        if constexpr (DECAY) {
          // S' decayed over the chunk; the keys of this wave's columns weighted
          // e^{gamma_C - gamma_j} (k slot e of kb[nt][q] is token 32 q + 8 g + e)
          const float eC = sEg[C - 1], gC = sGm[C - 1];
#pragma unroll
          for (int nt = 0; nt < NNT; ++nt) {
#pragma unroll
            for (int mt = 0; mt < NMT; ++mt) S[nt][mt] *= eC;
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
              for (int e = 0; e < 8; ++e)
                set_frag_elem(kb[nt][q], e, frag_elem(kb[nt][q], e) * __expf(gC - sGm[32 * q + 8 * g_ + e]));
          }
        }
        constexpr int G = 2, NG = NMT / G;
        Frag<T> ka[2][2 * G];
        auto load_group = [&](Frag<T>(&f)[2 * G], int g) {
#pragma unroll
          for (int e = 0; e < G; ++e)
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const int mt = G * g + e;
              f[2 * e + q] = frag_tr_any(ptr_pair + 32 * q * LDK + 32 * (mt >> 1) + 4 * (mt & 1), LDK);
            }
        };
        load_group(ka[0], 0);
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          if (g + 1 < NG) load_group(ka[(g + 1) & 1], g + 1);
          if constexpr (kDma) {
            if (g + 1 < NG) lds_wait_but<4 * G>(ka[g & 1]);
            else lds_wait(ka[g & 1]);
          }
#pragma unroll
          for (int e = 0; e < G; ++e)
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
              for (int nt = 0; nt < NNT; ++nt) mma(S[nt][G * g + e], ka[g & 1][2 * e + q], kb[nt][q]);
        }
      }
    }
    if constexpr (kDma) wait_vm_all();
    lds_barrier();  // (4) q_clean of chunk c complete, next chunk arrived; x, K', scores released
  }

  // copy out the last chunk
  {
    const int r0 = (cend - 1) * C, nrow = min(C, sq.len - r0);
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int e = tid + NT * u, row = e / VPR, col = (e % VPR) * 8;
      if (row < nrow)
        *reinterpret_cast<vec_t*>(qc + seq_off(sw, r0 + row, h, a.H, DK) + col) =
            *reinterpret_cast<const vec_t*>(sX + row * LDK + col);
    }
  }
}

namespace {
// The decay-aligned forms (a.la set) run forward only: no initial statistics,
// no training outputs of the contraction (base, m . x).
template <typename T, int DK>
hipError_t run_gram(const CleanArgs& a, hipStream_t st) {
  const long long nblk = (long long)a.B * a.H * n_segs(a.T, a.seg);
  if (nblk == 0) return hipSuccess;
  if (a.la && !a.sdec) return hipErrorInvalidValue;
  if (a.la)
    hipLaunchKernelGGL((clean_gram_kernel<T, DK, true>), dim3((unsigned)nblk), dim3(64 * (DK >= 128 ? 8 : 4)),
                       0, st, a);
  else
    hipLaunchKernelGGL((clean_gram_kernel<T, DK, false>), dim3((unsigned)nblk), dim3(64 * (DK >= 128 ? 8 : 4)),
                       0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_prefix(const CleanArgs& a, hipStream_t st) {
  const long long nblk = (long long)a.B * a.H * (DK * DK / 1024);
  if (nblk == 0) return hipSuccess;
  if (a.la && (a.t0 != 0 || a.C0 || a.mu0 || !a.sdec)) return hipErrorInvalidValue;
  if (a.la) hipLaunchKernelGGL((clean_prefix_kernel<T, DK, true>), dim3((unsigned)nblk), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((clean_prefix_kernel<T, DK, false>), dim3((unsigned)nblk), dim3(256), 0, st, a);
  return hipGetLastError();
}
template <typename T, int DK>
hipError_t run_out(const CleanArgs& a, hipStream_t st) {
  const long long nblk = (long long)a.B * a.H * n_segs(a.T, a.seg);
  if (nblk == 0) return hipSuccess;
  constexpr int NW = DK >= 128 ? 8 : 4;
  const bool train = a.base || a.corr || a.mdot || a.qclean_dbg;
  if (a.la) {
    if (a.base || a.mdot || a.t0 != 0 || a.mu0 || !a.sdec) return hipErrorInvalidValue;
    if (train)
      hipLaunchKernelGGL((clean_out_kernel<T, DK, NW, true, true>), dim3((unsigned)nblk), dim3(64 * NW), 0, st, a);
    else
      hipLaunchKernelGGL((clean_out_kernel<T, DK, NW, false, true>), dim3((unsigned)nblk), dim3(64 * NW), 0, st, a);
  } else if (train) {
    hipLaunchKernelGGL((clean_out_kernel<T, DK, NW, true, false>), dim3((unsigned)nblk), dim3(64 * NW), 0, st, a);
  } else {
    hipLaunchKernelGGL((clean_out_kernel<T, DK, NW, false, false>), dim3((unsigned)nblk), dim3(64 * NW), 0, st, a);
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
