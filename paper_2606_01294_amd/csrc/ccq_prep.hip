// ccq_prep.hip -- per-layer pre-processing of the raw queries and keys (Alg. 1:
// the l2 normalisation of Q and K and the gate Lambda = sigma(Q W_lambda^T + b_lambda)
// from the query before the head split; Eq. clean for the gate).
//
// Each wave takes four tokens: it requests their whole q and k rows at once
// (16-byte pieces, consecutive lanes along the row), reduces each head's
// squared norms over the aligned lane group holding that head and writes the
// normalised pieces; then every gate's partial dot products
// z[h'] += W[h'][j] q[j] over the lane's pieces, each piece of W read from LDS
// once for the four tokens; the H partial dots are reduced over the wave and
// lane h' writes lambda[h'].  Without output rows (q and k
// null) the kernel writes the row scales 1 / max(|x|, 1e-12) instead, for a
// forward that normalises as it stages the raw rows.  W (H x H dk, fp32) is staged
// in LDS once per workgroup and shared by its 16 tokens.  A wave reads each raw row before it writes the
// normalised one, so the outputs may overwrite the inputs.
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

namespace {
constexpr int kPrepTokens = 16;  // tokens per workgroup (4 per wave)
}  // namespace

// Sum over aligned groups of N consecutive lanes (N = 8, 16, 32), every lane
// receiving its group's sum.
template <int N>
__device__ __forceinline__ float lane_group_sum(float x) {
#pragma unroll
  for (int off = 1; off < N; off <<= 1) x += __shfl_xor(x, off);
  return x;
}

template <typename T, int DK, int HMAX>
__global__ __launch_bounds__(kThreads) void prep_kernel(const PrepArgs a) {
  extern __shared__ float sW[];  // [H][H * DK], each row split in half-pieces (below)
  constexpr int PPH = DK / 8;    // 8-element pieces per head row
  constexpr int NPMAX = 4;       // pieces per lane and token (H * DK <= 2048 when supported)
  typedef T v8 __attribute__((ext_vector_type(8)));
  const int H = a.H, E = H * DK, NP = E / 8;
  {  // W_lambda into LDS: every 16-byte piece requested before any is stored
    constexpr int NW4 = (int)(kPrepMaxLds / 16 / kThreads);
    const int n4 = H * E / 4;
    f32x4 wv[NW4];
#pragma unroll
    for (int u = 0; u < NW4; ++u) {
      const int i4 = threadIdx.x + kThreads * u;
      if (i4 < n4) wv[u] = reinterpret_cast<const f32x4*>(a.w)[i4];
    }
    // row g, features 8 p .. 8 p + 3 at g E + 4 p and 8 p + 4 .. 8 p + 7 at
    // g E + E / 2 + 4 p: a lane's two 16-byte reads of its piece p then sit
    // next to those of the neighbouring lanes (no bank conflicts)
#pragma unroll
    for (int u = 0; u < NW4; ++u) {
      const int i4 = threadIdx.x + kThreads * u;
      if (i4 < n4) {
        const int g = i4 / (E / 4), r = i4 % (E / 4);
        reinterpret_cast<f32x4*>(sW)[(g * E + (r & 1) * (E / 2)) / 4 + (r >> 1)] = wv[u];
      }
    }
  }
  __syncthreads();
  const int w = wave_id(), l = lane_id();
  const long long ntok = (long long)a.B * a.T;
  const T* qr = static_cast<const T*>(a.q_raw);
  const T* kr = static_cast<const T*>(a.k_raw);
  T* qo = static_cast<T*>(a.q);
  T* ko = static_cast<T*>(a.k);
  constexpr int TPW = kPrepTokens / 4;  // tokens per wave
  // every piece of the wave's tokens requested first
  v8 qa[TPW][NPMAX], ka[TPW][NPMAX];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const long long tok = (long long)blockIdx.x * kPrepTokens + w * TPW + tt;
#pragma unroll
    for (int i = 0; i < NPMAX; ++i) {
      const int p = l + 64 * i;
      if (tok < ntok && p < NP) {
        qa[tt][i] = *reinterpret_cast<const v8*>(qr + (size_t)tok * E + 8 * p);
        ka[tt][i] = *reinterpret_cast<const v8*>(kr + (size_t)tok * E + 8 * p);
      }
    }
  }
  // norms of every token's head rows; normalised rows (or the row scales) out
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const long long tok = (long long)blockIdx.x * kPrepTokens + w * TPW + tt;
    if (tok >= ntok) break;
    const size_t base = (size_t)tok * E;
#pragma unroll
    for (int i = 0; i < NPMAX; ++i) {
      const int p = l + 64 * i;
      float qf[8], kf[8], qq = 0.f, kk = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qf[e] = p < NP ? f32(qa[tt][i][e]) : 0.f;
        kf[e] = p < NP ? f32(ka[tt][i][e]) : 0.f;
        qq += qf[e] * qf[e];
        kk += kf[e] * kf[e];
      }
      // the lanes of one head row are an aligned group of PPH (or all 64 when PPH > 64)
      qq = lane_group_sum<(PPH < 64 ? PPH : 64)>(qq);
      kk = lane_group_sum<(PPH < 64 ? PPH : 64)>(kk);
      if (p < NP) {
        const float iq = 1.f / fmaxf(sqrtf(qq), 1e-12f), ik = 1.f / fmaxf(sqrtf(kk), 1e-12f);
        if (qo) {
          v8 yq, yk;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            yq[e] = to<T>(qf[e] * iq);
            yk[e] = to<T>(kf[e] * ik);
          }
          *reinterpret_cast<v8*>(qo + base + 8 * p) = yq;
          *reinterpret_cast<v8*>(ko + base + 8 * p) = yk;
        } else if (p % PPH == 0) {  // the row scales instead, from the head's first lane
          a.rq[(size_t)tok * H + p / PPH] = iq;
          a.rk[(size_t)tok * H + p / PPH] = ik;
        }
      }
    }
  }
  // the gates: every W piece read from LDS serves all TPW tokens of the wave
  float z[TPW][HMAX];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
    for (int g = 0; g < HMAX; ++g) z[tt][g] = 0.f;
#pragma unroll
  for (int i = 0; i < NPMAX; ++i) {
    const int p = l + 64 * i;
    if (p < NP) {
      float qf[TPW][8];
#pragma unroll
      for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[tt][e] = f32(qa[tt][i][e]);
#pragma unroll
      for (int g = 0; g < HMAX; ++g) {
        if (g < H) {
          const f32x4 w0 = *reinterpret_cast<const f32x4*>(sW + g * E + 4 * p);
          const f32x4 w1 = *reinterpret_cast<const f32x4*>(sW + g * E + E / 2 + 4 * p);
#pragma unroll
          for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
            for (int e = 0; e < 4; ++e) z[tt][g] += w0[e] * qf[tt][e] + w1[e] * qf[tt][4 + e];
        }
      }
    }
  }
  // sums over the wave of the TPW x HMAX partial dots by a reduce-scatter
  // butterfly: at each step a lane keeps half of its values, adds its
  // partner's copy of them and hands over the other half, so that after
  // log2(TPW HMAX) steps lane l holds the partial sum of value l % (TPW HMAX)
  // over the lanes that share its low bits; one more exchange (when 64 lanes
  // exceed the values) completes the sum
  constexpr int NZ = TPW * HMAX;  // 64
  static_assert(NZ == 64, "one value per lane after the butterfly");
  float zz[NZ];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
    for (int g = 0; g < HMAX; ++g) zz[tt * HMAX + g] = z[tt][g];
#pragma unroll
  for (int half = NZ / 2; half >= 1; half >>= 1) {
    // lanes with bit `half` set keep the upper half of their current values
    const bool up = (l & half) != 0;
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const float mine = up ? zz[half + j] : zz[j];
      const float other = up ? zz[j] : zz[half + j];
      zz[j] = mine + __shfl_xor(other, half);
    }
  }
  // lane l now holds value l (token l / HMAX, gate l % HMAX), summed over the wave
  {
    const int tt = l / HMAX, g = l % HMAX;
    const long long tok = (long long)blockIdx.x * kPrepTokens + w * TPW + tt;
    if (g < H && tok < ntok) a.lam[(size_t)tok * H + g] = 1.f / (1.f + __expf(-(zz[0] + a.b[g])));
  }
}

namespace {
template <typename T, int DK>
hipError_t run_prep(const PrepArgs& a, hipStream_t st) {
  const long long ntok = (long long)a.B * a.T;
  if (ntok == 0 || a.H == 0) return hipSuccess;
  const unsigned nblk = (unsigned)((ntok + kPrepTokens - 1) / kPrepTokens);
  const size_t lds = (size_t)a.H * a.H * DK * sizeof(float);
  hipLaunchKernelGGL((prep_kernel<T, DK, kPrepMaxHeads>), dim3(nblk), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}
template <typename T>
hipError_t prep_dispatch(const PrepArgs& a, hipStream_t st) {
  switch (a.dk) {
    case 64: return run_prep<T, 64>(a, st);
    case 128: return run_prep<T, 128>(a, st);
    case 256: return run_prep<T, 256>(a, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

bool prep_supported(int H, int dk) {
  // H * dk <= 2048 follows from the LDS bound for H >= 8; it is checked for
  // fewer heads too (at most four 8-element pieces per lane and token)
  return (dk == 64 || dk == 128 || dk == 256) && H >= 1 && H <= kPrepMaxHeads &&
         (size_t)H * H * dk * sizeof(float) <= kPrepMaxLds && H * dk <= 2048;
}

hipError_t launch_prep(const PrepArgs& a, bool is_bf16, hipStream_t st) {
  return is_bf16 ? prep_dispatch<bf16_t>(a, st) : prep_dispatch<float>(a, st);
}

}  // namespace ccq
