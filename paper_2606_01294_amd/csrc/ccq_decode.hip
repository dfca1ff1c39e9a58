// ccq_decode.hip -- one recurrent CCQ step per sequence (Alg. 2, recurrent
// inference) on the cache triple (S, Cbar, mu), updated in place.
//
// With t the 1-based position of the new token (t0 + 1):
//   Cbar_t = Cbar_{t-1} + (k k^T - Cbar_{t-1}) / t,   mu_t = mu_{t-1} + (k - mu_{t-1}) / t,
//   Sigma_t q = Cbar_t q - mu_t (mu_t . q)          (Cbar_t q alone when uncentred),
//   q_clean = q - lam Sigma_t q,
//   S_t = BackboneUpdate(S_{t-1}; k, v, gates),      o = scale S_t q_clean.
// Both backbone writes act on each row of S on its own (GLA: S[r] e^g + v_r k;
// Gated DeltaNet: alpha S[r] - alpha beta (S[r] . k) k + beta v_r k), and
// q_clean needs only the head's own Cbar and mu, so one workgroup can carry
// a head through the whole step (decode_kernel, one launch, no workspace);
// for a few large heads the step is split over 16-row blocks in two launches
// (decode_cbar_kernel, decode_s_kernel).
#include "ccq_device.h"
#include "ccq_kernels.h"

namespace ccq {

namespace {
constexpr int kDecThreads = 1024;            // one workgroup per (sequence, head)
constexpr int kDecTpr = 16;                  // threads per cache row
constexpr int kDecRps = kDecThreads / kDecTpr;  // rows per sweep (64)
constexpr int kDecRegs = 16;                 // f32x4 of Cbar held per thread at most
constexpr int kDecBatch = 8;                 // f32x4 of S per thread and batch (two in flight)

template <typename T>
__device__ __forceinline__ float ldf(const void* p, size_t i) {
  return static_cast<float>(static_cast<const T*>(p)[i]);
}
// Every sweep reads the same columns of q, k and q_clean from LDS; reading
// them again per sweep (a few ds_read_b128) is cheaper than holding them in
// registers beside the cache pieces, so the compiler is kept from merging the
// reads across sweeps.
__device__ __forceinline__ void reread_lds() { asm volatile("" ::: "memory"); }

// Loads of one head's cache matrix go through a raw buffer (bounds-checked
// by the hardware against its byte size): one VGPR of per-thread offset
// serves every load, the sweep's offset going in an SGPR and the piece's in
// the instruction's immediate.  Stores are global stores of the same form
// (uniform 64-bit base, 32-bit per-thread offset): with a buffer store whose
// offset sits in an SGPR, the compiler does not separate the store from a
// following write of its data registers, and the store was seen to take the
// new value in some lanes.
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc head_rsrc(float* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(p, 0, bytes, 0x00020000);
}
__device__ __forceinline__ f32x4 bload(Rsrc r, int voff, int soff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ void gstore(const f32x4& x, float* base, unsigned off_bytes) {
  *reinterpret_cast<f32x4*>(reinterpret_cast<char*>(base) + off_bytes) = x;
}
}  // namespace

// The whole step for one (sequence, head) in one workgroup of 1024 threads.
// A cache row of DK fp32 is read by 16 consecutive threads, thread j taking
// the 16-byte pieces j, j + 16, ... (so each load instruction of a wave reads
// 4 rows x 256 contiguous bytes), and a sweep covers 64 rows.
//   1. the DK rows of Cbar, updated, with (Cbar_t q)[n] summed over each
//      row's threads; mu_t and mu_t . q;
//   2. q_clean into LDS;
//   3. the DV rows of S in batches of at most kDecBatch f32x4 per thread, the
//      next batch loading while one is worked on: the
//      backbone write and the read o_r = scale S_t[r] . q_clean.
// Every cache element is read once and written once.  The first batch of S
// is loaded beside Cbar when both fit in registers, else as soon as Cbar is
// stored, so that its latency overlaps the reductions of steps 1 and 2.
template <typename T, typename TG, int DK, int DV, bool GDN>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(const DecodeArgs a) {
  constexpr int NV = DK / (4 * kDecTpr);       // f32x4 per thread and row
  constexpr int NSC = DK / kDecRps;            // sweeps over Cbar
  constexpr int NSS = DV / kDecRps;            // sweeps over S
  constexpr int NB = NSS < kDecBatch / NV ? NSS : kDecBatch / NV;  // S sweeps per batch
  constexpr int NBATCH = NSS / NB;
  constexpr bool EARLY = (NSC + NB) * NV <= kDecRegs;
  static_assert(NV >= 1 && NSC * NV <= kDecRegs && NSS % NB == 0, "decode shape");
  __shared__ __align__(16) float sQ[DK], sK[DK], sE[DK], sCq[DK], sMu[DK], sQc[DK];
  __shared__ float sRed[kDecThreads / 64];
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int j = tid % kDecTpr, rr = tid / kDecTpr;
  const size_t tb = (size_t)bh * DK, vb = (size_t)bh * DV;
  const float inv_t = 1.f / (float)(a.t0 + 1);
  auto col = [&](int i, int e) { return 4 * (i * kDecTpr + j) + e; };
  float* const Ch = a.C + tb * DK;
  float* const Sh = a.S + vb * DK;
  const Rsrc rC = head_rsrc(Ch, DK * DK * 4), rS = head_rsrc(Sh, DV * DK * 4);
  const int voff = (rr * DK + 4 * j) * 4;  // bytes; + 256 i for piece i, + sweep * 64 DK * 4
  constexpr int kSweep = kDecRps * DK * 4;

  f32x4 xc[NSC][NV], xs[2][NB][NV];
  auto load_s = [&](int batch) {
#pragma unroll
    for (int w = 0; w < NB; ++w)
#pragma unroll
      for (int i = 0; i < NV; ++i)
        xs[batch & 1][w][i] = bload(rS, voff + 256 * i, (batch * NB + w) * kSweep);
  };
#pragma unroll
  for (int w = 0; w < NSC; ++w)
#pragma unroll
    for (int i = 0; i < NV; ++i)
      xc[w][i] = bload(rC, voff + 256 * i, w * kSweep);
  if constexpr (EARLY) load_s(0);
  for (int c = tid; c < DK; c += kDecThreads) {
    sQ[c] = ldf<T>(a.q, tb + c);
    sK[c] = ldf<T>(a.k, tb + c);
    if constexpr (!GDN) sE[c] = __expf(ldf<TG>(a.g, tb + c));
  }
  __syncthreads();

  // 1. Cbar_t = Cbar + (k k^T - Cbar) / t and Cbar_t q
  float cq[NSC];
#pragma unroll
  for (int w = 0; w < NSC; ++w) {
    reread_lds();
    const float kn = sK[w * kDecRps + rr];
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xc[w][i][e] += (kn * sK[col(i, e)] - xc[w][i][e]) * inv_t;
        acc += xc[w][i][e] * sQ[col(i, e)];
      }
    // the sum is formed here, so that the pieces are free once stored
    asm volatile("" : "+v"(acc));
    cq[w] = acc;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      gstore(xc[w][i], Ch + w * (kSweep / 4), voff + 256 * i);
  }
  if constexpr (!EARLY) {
    reread_lds();
    load_s(0);
  }
#pragma unroll
  for (int w = 0; w < NSC; ++w) {
    const float acc = group_sum<kDecTpr>(cq[w]);
    if (j == 0) sCq[w * kDecRps + rr] = acc;
  }
  // mu_t = mu + (k - mu) / t and mu_t . q
  float mq = 0.f;
  for (int c = tid; c < DK; c += kDecThreads) {
    const float m0 = a.mu[tb + c];
    const float m = m0 + (sK[c] - m0) * inv_t;
    a.mu[tb + c] = m;
    sMu[c] = m;
    mq += m * sQ[c];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mq += __shfl_xor(mq, off);
  if ((tid & 63) == 0) sRed[tid >> 6] = mq;
  __syncthreads();

  // 2. q_clean = q - lam (Cbar_t q - mu_t (mu_t . q))   (Cbar_t q alone when uncentred)
  mq = 0.f;
#pragma unroll
  for (int w = 0; w < kDecThreads / 64; ++w) mq += sRed[w];
  const float lam = a.lam[bh];
  for (int c = tid; c < DK; c += kDecThreads)
    sQc[c] = sQ[c] - lam * (sCq[c] - (a.centered ? sMu[c] * mq : 0.f));
  __syncthreads();

  // 3. rows of S: the backbone write, then o_r
  float alpha = 1.f, bt = 0.f, kq = 0.f;
  if constexpr (GDN) {
    alpha = __expf(static_cast<const float*>(a.g)[bh]);
    bt = a.beta[bh];
    // k . q_clean, the same for every row
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) kq += sK[col(i, e)] * sQc[col(i, e)];
    kq = group_sum<kDecTpr>(kq);
  }
#pragma unroll
  for (int batch = 0; batch < NBATCH; ++batch) {
    if (batch + 1 < NBATCH) load_s(batch + 1);
    f32x4 (&x)[NB][NV] = xs[batch & 1];
#pragma unroll
    for (int w = 0; w < NB; ++w) {
      reread_lds();
      const int r = (batch * NB + w) * kDecRps + rr;
      const float vr = ldf<T>(a.v, vb + r);
      float o = 0.f;
      if constexpr (GDN) {
        // o_r = alpha S_{t-1}[r] . q_clean + coef (k . q_clean) with
        // coef = beta (v_r - alpha S_{t-1}[r] . k)
        float y = 0.f, z = 0.f;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          reread_lds();
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            y += x[w][i][e] * sK[col(i, e)];
            z += x[w][i][e] * sQc[col(i, e)];
          }
        }
        y = group_sum<kDecTpr>(y);
        z = group_sum<kDecTpr>(z);
        const float coef = bt * (vr - alpha * y);
        o = alpha * z + coef * kq;
        reread_lds();
#pragma unroll
        for (int i = 0; i < NV; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) x[w][i][e] = alpha * x[w][i][e] + coef * sK[col(i, e)];
      } else {
#pragma unroll
        for (int i = 0; i < NV; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x[w][i][e] = x[w][i][e] * sE[col(i, e)] + vr * sK[col(i, e)];
            o += x[w][i][e] * sQc[col(i, e)];
          }
        o = group_sum<kDecTpr>(o);
      }
#pragma unroll
      for (int i = 0; i < NV; ++i)
        gstore(x[w][i], Sh + (batch * NB + w) * (kSweep / 4), voff + 256 * i);
      if (j == 0) static_cast<T*>(a.o)[vb + r] = static_cast<T>(a.scale * o);
    }
  }
}

// For batches too small to fill the chip with one workgroup per head, the
// step is two launches over blocks of 16 cache rows (one 256-thread
// workgroup each, a row read by 16 consecutive threads as above), the
// launch boundary carrying Cbar_t q from the first to the second:
//   decode_cbar_kernel: 16 rows of Cbar updated and (Cbar_t q)[n] of those
//     rows to the workspace; the first block of a head also updates mu;
//   decode_s_kernel: 16 rows of S loaded first, then q_clean formed from
//     Cbar_t q and mu_t, then the backbone write and o_r = scale S_t[r] .
//     q_clean.
constexpr int kPartThreads = 256;
constexpr int kPartRows = kPartThreads / kDecTpr;  // 16

template <typename T, int DK>
__global__ __launch_bounds__(kPartThreads) void decode_cbar_kernel(const DecodeArgs a) {
  constexpr int NV = DK / (4 * kDecTpr);
  __shared__ __align__(16) float sQ[DK], sK[DK];
  const int blk = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int j = tid % kDecTpr, rr = tid / kDecTpr;
  const size_t tb = (size_t)bh * DK;
  const float inv_t = 1.f / (float)(a.t0 + 1);
  auto col = [&](int i, int e) { return 4 * (i * kDecTpr + j) + e; };
  float* const Cb = a.C + (tb + blk * kPartRows) * DK;
  const Rsrc rC = head_rsrc(Cb, kPartRows * DK * 4);
  const int voff = (rr * DK + 4 * j) * 4;
  f32x4 x[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] = bload(rC, voff + 256 * i, 0);
  for (int c = tid; c < DK; c += kPartThreads) {
    sQ[c] = ldf<T>(a.q, tb + c);
    sK[c] = ldf<T>(a.k, tb + c);
  }
  __syncthreads();
  const int n = blk * kPartRows + rr;
  const float kn = sK[n];
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[i][e] += (kn * sK[col(i, e)] - x[i][e]) * inv_t;
      acc += x[i][e] * sQ[col(i, e)];
    }
#pragma unroll
  for (int i = 0; i < NV; ++i) gstore(x[i], Cb, voff + 256 * i);
  acc = group_sum<kDecTpr>(acc);
  if (j == 0) a.cq[tb + n] = acc;
  if (blk == 0)
    for (int c = tid; c < DK; c += kPartThreads) {
      const float m0 = a.mu[tb + c];
      a.mu[tb + c] = m0 + (sK[c] - m0) * inv_t;
    }
}

template <typename T, typename TG, int DK, int DV, bool GDN>
__global__ __launch_bounds__(kPartThreads) void decode_s_kernel(const DecodeArgs a) {
  constexpr int NV = DK / (4 * kDecTpr);
  __shared__ __align__(16) float sK[DK], sE[DK], sQc[DK];
  __shared__ float sRed[kPartThreads / 64];
  const int blk = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int j = tid % kDecTpr, rr = tid / kDecTpr;
  const size_t tb = (size_t)bh * DK, vb = (size_t)bh * DV;
  auto col = [&](int i, int e) { return 4 * (i * kDecTpr + j) + e; };
  float* const Sb = a.S + (vb + blk * kPartRows) * DK;
  const Rsrc rS = head_rsrc(Sb, kPartRows * DK * 4);
  const int voff = (rr * DK + 4 * j) * 4;
  f32x4 x[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] = bload(rS, voff + 256 * i, 0);
  const int r = blk * kPartRows + rr;
  const float vr = ldf<T>(a.v, vb + r);

  // q_clean = q - lam (Cbar_t q - mu_t (mu_t . q))   (Cbar_t q alone when uncentred)
  float q = 0.f, cq = 0.f, mu = 0.f, mq = 0.f;
  if (tid < DK) {
    q = ldf<T>(a.q, tb + tid);
    cq = a.cq[tb + tid];
    mu = a.mu[tb + tid];
    mq = mu * q;
    sK[tid] = ldf<T>(a.k, tb + tid);
    if constexpr (!GDN) sE[tid] = __expf(ldf<TG>(a.g, tb + tid));
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mq += __shfl_xor(mq, off);
  if ((tid & 63) == 0) sRed[tid >> 6] = mq;
  __syncthreads();
  mq = 0.f;
#pragma unroll
  for (int w = 0; w < kPartThreads / 64; ++w) mq += sRed[w];
  if (tid < DK) sQc[tid] = q - a.lam[bh] * (cq - (a.centered ? mu * mq : 0.f));
  __syncthreads();

  float o = 0.f;
  if constexpr (GDN) {
    const float alpha = __expf(static_cast<const float*>(a.g)[bh]), bt = a.beta[bh];
    float y = 0.f;  // S_{t-1}[r] . k
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) y += x[i][e] * sK[col(i, e)];
    y = group_sum<kDecTpr>(y);
    const float coef = bt * (vr - alpha * y);
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[i][e] = alpha * x[i][e] + coef * sK[col(i, e)];
        o += x[i][e] * sQc[col(i, e)];
      }
  } else {
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[i][e] = x[i][e] * sE[col(i, e)] + vr * sK[col(i, e)];
        o += x[i][e] * sQc[col(i, e)];
      }
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) gstore(x[i], Sb, voff + 256 * i);
  o = group_sum<kDecTpr>(o);
  if (j == 0) static_cast<T*>(a.o)[vb + r] = static_cast<T>(a.scale * o);
}

namespace {
template <typename T, typename TG, int DK, int DV, bool GDN>
hipError_t run_decode_g(const DecodeArgs& a, hipStream_t st) {
  const int bh = a.B * a.H;
  if (!decode_split(bh, DK, DV)) {
    hipLaunchKernelGGL((decode_kernel<T, TG, DK, DV, GDN>), dim3(bh), dim3(kDecThreads), 0, st, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((decode_cbar_kernel<T, DK>), dim3(DK / kPartRows, bh), dim3(kPartThreads), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_s_kernel<T, TG, DK, DV, GDN>), dim3(DV / kPartRows, bh), dim3(kPartThreads), 0, st, a);
  return hipGetLastError();
}
template <typename T, typename TG, int DK, int DV>
hipError_t run_decode_v(const DecodeArgs& a, bool gdn, hipStream_t st) {
  if (a.B * a.H == 0) return hipSuccess;
  return gdn ? run_decode_g<T, float, DK, DV, true>(a, st) : run_decode_g<T, TG, DK, DV, false>(a, st);
}
template <typename T, typename TG, int DK>
hipError_t run_decode(const DecodeArgs& a, bool gdn, hipStream_t st) {
  switch (a.dv) {
    case 64: return run_decode_v<T, TG, DK, 64>(a, gdn, st);
    case 128: return run_decode_v<T, TG, DK, 128>(a, gdn, st);
    case 256: return run_decode_v<T, TG, DK, 256>(a, gdn, st);
    case 512: return run_decode_v<T, TG, DK, 512>(a, gdn, st);
  }
  return hipErrorInvalidValue;
}
template <typename T, typename TG>
hipError_t decode_dispatch(const DecodeArgs& a, bool gdn, hipStream_t st) {
  switch (a.dk) {
    case 64: return run_decode<T, TG, 64>(a, gdn, st);
    case 128: return run_decode<T, TG, 128>(a, gdn, st);
    case 256: return run_decode<T, TG, 256>(a, gdn, st);
  }
  return hipErrorInvalidValue;
}
}  // namespace

// One workgroup per head is bounded by what one compute unit moves (about
// 88 GB/s for this stream of loads and stores, after about 5 us of launch and
// latency); the two launches over 16-row blocks spread the cache over the
// whole chip but cost about 8 us fixed.  Both figures are measured on MI355X
// (one workgroup per head: 9.5 us for 384 KB of cache traffic per head, 16.8 us
// for 1 MB; the split: 10.4 and 11.7 us for 32 such heads).  Under 256 heads
// the step takes whichever model says is faster; from 256 heads on, one
// workgroup per head fills the chip.
bool decode_split(long long bh, int dk, int dv) {
  if (bh >= 256) return false;
  const double per_head = 8.0 * ((double)dk * dk + (double)dv * dk);  // bytes read and written
  const double t_single = 5.1e-6 + per_head / 88e9;
  const double t_split = 8.0e-6 + per_head * (double)bh / 5e12;
  return t_split < t_single;
}

bool decode_supported(int dk, int dv) {
  return (dk == 64 || dk == 128 || dk == 256) && (dv == 64 || dv == 128 || dv == 256 || dv == 512);
}

hipError_t launch_decode(const DecodeArgs& a, bool gdn, bool is_bf16, bool gate_bf16, hipStream_t st) {
  if (is_bf16)
    return gate_bf16 ? decode_dispatch<bf16_t, bf16_t>(a, gdn, st) : decode_dispatch<bf16_t, float>(a, gdn, st);
  return gate_bf16 ? decode_dispatch<float, bf16_t>(a, gdn, st) : decode_dispatch<float, float>(a, gdn, st);
}

}  // namespace ccq
