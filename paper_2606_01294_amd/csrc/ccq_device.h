// ccq_device.h -- device helpers shared by the CCQ kernels (gfx950 / CDNA4).
//
// Matrix products use the 16x16 MFMA tile with fp32 accumulation:
//   bf16: v_mfma_f32_16x16x32_bf16  (one instruction per 32-wide k step)
//   fp32: v_mfma_f32_16x16x4_f32    (eight instructions per 32-wide k step)
// A "fragment" is the 8 consecutive contraction elements one lane feeds per
// 32-wide k step: lane l supplies row (l % 16) of the A tile and column
// (l % 16) of the B tile, k = 8*(l / 16) .. 8*(l / 16) + 7.  For fp32 the
// eight sub-steps walk those same eight k values, so both dtypes read the
// same LDS bytes per lane.  The accumulator holds D[4*(l/16) + r][l % 16] in
// element r.  B tiles are kept in LDS as B^T (row = output column, k
// contiguous) so that every fragment is one contiguous 16-byte (bf16) or
// 32-byte (fp32) LDS read.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace ccq {

constexpr int kChunk = 64;    // chunk length C of the chunkwise form
constexpr int kThreads = 256; // four 64-wide waves per workgroup
constexpr int kOutThreads = 512;  // eight waves: chunk-parallel output kernels

// The 16 16x16 tiles of a 64x64 chunk block, lower ones (I >= J) first:
// tile t < 10 is (I, J) with J <= I, tiles 10..15 are the upper ones.
__device__ __forceinline__ int intra_tile_row(int t) { return (int)((0x940ffa94ull >> (2 * t)) & 3); }
__device__ __forceinline__ int intra_tile_col(int t) { return (int)((0xfb9e4910ull >> (2 * t)) & 3); }

template <typename T>
struct Pad { static constexpr int value = 32 / (int)sizeof(T); };  // 32-byte row padding

template <typename T> struct Frag;
template <> struct Frag<bf16_t> { bf16x8 v; };
template <> struct Frag<float> { f32x4 lo, hi; };

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// Fragment of a 16-row tile stored row-major in LDS with leading dimension ld
// (elements); `tile` points at (row 0, k0).
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag(const T* tile, int ld) {
  const int l = lane_id();
  const T* p = tile + (l & 15) * ld + 8 * (l >> 4);
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    f.v = *reinterpret_cast<const bf16x8*>(p);
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(p);
    f.hi = *reinterpret_cast<const f32x4*>(p + 4);
  }
  return f;
}

// Same fragment read straight from global memory (row pitch ld elements).
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag_global(const T* tile, size_t ld) {
  const int l = lane_id();
  const T* p = tile + (size_t)(l & 15) * ld + 8 * (l >> 4);
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    f.v = *reinterpret_cast<const bf16x8*>(p);
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(p);
    f.hi = *reinterpret_cast<const f32x4*>(p + 4);
  }
  return f;
}

// Fragment of a transposed operand: element (m, k) of the MFMA operand is
// X[k][m] of a row-major LDS tile X (k runs along X's rows).  `base` points at
// X[k0][m0], ld is X's row pitch in elements (a multiple of 4).  For bf16 this
// uses the gfx950 transposing LDS read: within each 16-lane group, lane j
// addresses row k0 + 8g + j/4, column m0 + 4 (j % 4), and lane i receives
// X[k0 + 8g .. + 3][m0 + i]; a second read covers the next four rows.
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag_tr(const T* base, int ld);

template <>
__device__ __forceinline__ Frag<bf16_t> ld_frag_tr<bf16_t>(const bf16_t* base, int ld) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const bf16_t* p = base + (8 * g + (j >> 2)) * ld + 4 * (j & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * ld));
  Frag<bf16_t> f;
  f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return f;
}

template <>
__device__ __forceinline__ Frag<float> ld_frag_tr<float>(const float* base, int ld) {
  const int l = lane_id(), g = l >> 4, m = l & 15;
  Frag<float> f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f.lo[e] = base[(8 * g + e) * ld + m];
    f.hi[e] = base[(8 * g + 4 + e) * ld + m];
  }
  return f;
}

// Transposed-operand fragment whose k slots follow two stacked accumulator
// tiles (rows 0..15 and 16..31 of a 32-row block): slot 8g + e is row 4g + e
// for e < 4 and row 16 + 4g + (e - 4) otherwise.  Paired with
// acc_pair_frag, a product can consume a score tile straight from the
// accumulators of an earlier one, with no trip through LDS.  `base` points at
// X[k0][m0] of a row-major LDS tile with row pitch ld.
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag_tr_acc(const T* base, int ld);

template <>
__device__ __forceinline__ Frag<bf16_t> ld_frag_tr_acc<bf16_t>(const bf16_t* base, int ld) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const bf16_t* p = base + (4 * g + (j >> 2)) * ld + 4 * (j & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 16 * ld));
  Frag<bf16_t> f;
  f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return f;
}

template <>
__device__ __forceinline__ Frag<float> ld_frag_tr_acc<float>(const float* base, int ld) {
  const int l = lane_id(), g = l >> 4, m = l & 15;
  Frag<float> f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f.lo[e] = base[(4 * g + e) * ld + m];
    f.hi[e] = base[(16 + 4 * g + e) * ld + m];
  }
  return f;
}

// ld_frag_tr_acc with the fragment's 16 rows (X's columns) taken in pair
// order: fragment row m is column pair_col(t, m) = 32 (t / 2) + 8 (m / 4) +
// 4 (t % 2) + m % 4 of X for tile t of a 32-column block pair.  Accumulator
// tiles 2s and 2s + 1 formed from such operands hold, in lane group g, the 8
// consecutive columns 32 s + 8 g .. + 7, so acc_pair_frag packs them into an
// operand whose k slots are in natural order (read by plain ld_frag).  `base`
// points at X[k0][c0]; t is the 16-column tile index counted from c0 (c0 a
// multiple of 32).
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag_tr_acc_pair(const T* base, int ld, int t);

template <>
__device__ __forceinline__ Frag<bf16_t> ld_frag_tr_acc_pair<bf16_t>(const bf16_t* base, int ld, int t) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int l = lane_id(), g = l >> 4, j = l & 15;
  const bf16_t* p = base + (4 * g + (j >> 2)) * ld + 32 * (t >> 1) + 4 * (t & 1) + 8 * (j & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 16 * ld));
  Frag<bf16_t> f;
  f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return f;
}

template <>
__device__ __forceinline__ Frag<float> ld_frag_tr_acc_pair<float>(const float* base, int ld, int t) {
  const int l = lane_id(), g = l >> 4, m = l & 15;
  const int col = 32 * (t >> 1) + 4 * (t & 1) + 8 * (m >> 2) + (m & 3);
  Frag<float> f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f.lo[e] = base[(4 * g + e) * ld + col];
    f.hi[e] = base[(16 + 4 * g + e) * ld + col];
  }
  return f;
}

// Feature held in accumulator row 4 g + r of tile t of a pair-ordered state
// (ld_frag_tr_acc_pair): 32 (t / 2) + 8 g + 4 (t % 2) + r.
__host__ __device__ __forceinline__ int pair_feat(int t, int g) { return 32 * (t >> 1) + 8 * g + 4 * (t & 1); }

// Row-operand fragment in the same k-slot order as ld_frag_tr_acc: lane l
// reads row (l % 16) of a row-major tile at k = 4g .. 4g+3 and 16 + 4g ..
// 16 + 4g + 3 (g = l / 16).  `tile` points at (row 0, k0); works for LDS or
// global pointers.
template <typename T>
__device__ __forceinline__ Frag<T> ld_frag_acc(const T* tile, size_t ld) {
  const int l = lane_id(), g = l >> 4;
  const T* p = tile + (size_t)(l & 15) * ld + 4 * g;
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 16);
    f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(p);
    f.hi = *reinterpret_cast<const f32x4*>(p + 16);
  }
  return f;
}

// B fragment (k = accumulator row, n = accumulator column) built from two
// accumulator tiles: x holds rows 0..15, y rows 16..31 of the k range.
template <typename T>
__device__ __forceinline__ Frag<T> acc_pair_frag(const f32x4& x, const f32x4& y) {
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    f.v = bf16x8{static_cast<bf16_t>(x[0]), static_cast<bf16_t>(x[1]), static_cast<bf16_t>(x[2]),
                 static_cast<bf16_t>(x[3]), static_cast<bf16_t>(y[0]), static_cast<bf16_t>(y[1]),
                 static_cast<bf16_t>(y[2]), static_cast<bf16_t>(y[3])};
  } else {
    f.lo = x;
    f.hi = y;
  }
  return f;
}

// Storage position, within its 32-element block, that puts logical element c
// where an accumulator pair keeps it: lane group g holds logical 4g..4g+3 and
// 16+4g..16+4g+3, stored at 8g..8g+7.  A row written in this order is read
// back by ld_frag / ld_frag_global (8 contiguous elements) in the k-slot order
// of ld_frag_tr_acc / acc_pair_frag.
__host__ __device__ __forceinline__ int acc_pos(int c) {
  return (c & ~31) | (((c & 15) >> 2) << 3) | ((c & 16) >> 2) | (c & 3);
}
// Inverse of acc_pos: the logical element stored at position p.
__host__ __device__ __forceinline__ int acc_logical(int p) {
  return (p & ~31) | (((p >> 2) & 1) << 4) | (((p >> 3) & 3) << 2) | (p & 3);
}

// Store two accumulator tiles' lane values (x: logical 4g..4g+3, y: 16+4g..)
// as the 8 contiguous elements at p (acc_pos order): one 16- or 32-byte store.
template <typename T>
__device__ __forceinline__ void store_acc_pair(T* p, const f32x4& x, const f32x4& y) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<bf16x8*>(p) = acc_pair_frag<T>(x, y).v;
  } else {
    *reinterpret_cast<f32x4*>(p) = x;
    *reinterpret_cast<f32x4*>(p + 4) = y;
  }
}

template <typename T>
__device__ __forceinline__ float frag_elem(const Frag<T>& f, int e) {
  if constexpr (sizeof(T) == 2) {
    return static_cast<float>(f.v[e]);
  } else {
    return e < 4 ? f.lo[e] : f.hi[e - 4];
  }
}

template <typename T>
__device__ __forceinline__ void set_frag_elem(Frag<T>& f, int e, float x) {
  if constexpr (sizeof(T) == 2) {
    f.v[e] = static_cast<bf16_t>(x);
  } else {
    if (e < 4) f.lo[e] = x;
    else f.hi[e - 4] = x;
  }
}

// Store a fragment's 8 elements contiguously (one 16- or 32-byte store).
template <typename T>
__device__ __forceinline__ void store_frag(T* p, const Frag<T>& f) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<bf16x8*>(p) = f.v;
  } else {
    *reinterpret_cast<f32x4*>(p) = f.lo;
    *reinterpret_cast<f32x4*>(p + 4) = f.hi;
  }
}

// acc += A[16 x 16] B[16 x 16] in fp32 (four 16x16x4 steps), both operands
// row-major in LDS: A at a (pitch lda), B at b (pitch ldb, rows = k).
__device__ __forceinline__ void mma16_f32(f32x4& acc, const float* a, int lda, const float* b, int ldb) {
  const int l = lane_id(), g = l >> 4, m = l & 15;
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[m * lda + 4 * kk + g], b[(4 * kk + g) * ldb + m], acc, 0, 0, 0);
}

// B fragment of the 16-column tile whose column 0 is all ones (the rest zero):
// acc += A * ones gives the row sums of A in column 0.
template <typename T>
__device__ __forceinline__ Frag<T> ones_col_frag() {
  const T one = static_cast<T>((lane_id() & 15) == 0 ? 1.f : 0.f);
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    f.v = bf16x8{one, one, one, one, one, one, one, one};
  } else {
    f.lo = f32x4{one, one, one, one};
    f.hi = f.lo;
  }
  return f;
}

// Store the four accumulator values of this lane (rows 4g..4g+3 of the tile,
// one column) as four consecutive elements of row `col` of a row-major LDS
// array: the transposed tile, written with one 8- or 16-byte store.
template <typename T>
__device__ __forceinline__ void store4(T* p, float x0, float x1, float x2, float x3) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<bf16x4*>(p) = bf16x4{static_cast<bf16_t>(x0), static_cast<bf16_t>(x1),
                                           static_cast<bf16_t>(x2), static_cast<bf16_t>(x3)};
  } else {
    *reinterpret_cast<f32x4*>(p) = f32x4{x0, x1, x2, x3};
  }
}

__device__ __forceinline__ void mma(f32x4& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}

__device__ __forceinline__ void mma(f32x4& acc, const Frag<float>& a, const Frag<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[0], b.lo[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[1], b.lo[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[2], b.lo[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo[3], b.lo[3], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[0], b.hi[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[1], b.hi[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[2], b.hi[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi[3], b.hi[3], acc, 0, 0, 0);
}

// acc += A[16 x K] * B^T[16 x K]^T with both operands in LDS.
template <typename T, int K>
__device__ __forceinline__ void tile_mma(f32x4& acc, const T* a, int lda, const T* bt, int ldb) {
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += 32) mma(acc, ld_frag(a + k0, lda), ld_frag(bt + k0, ldb));
}

// The same product over the chunk index with operands in row-major chunk
// tiles (rows = the chunk's tokens): tile_mma_tr takes both operands with
// transposing LDS reads, acc += A[:, a0..]^T B[:, b0..] (at = A + a0,
// bt = B + b0); tile_mma_bt only the second, acc += A B for a 16-row block of
// A and a 16-column block of B (b = B + b0).
template <typename T, int K>
__device__ __forceinline__ void tile_mma_tr(f32x4& acc, const T* at, int lda, const T* bt, int ldb) {
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += 32) mma(acc, ld_frag_tr(at + k0 * lda, lda), ld_frag_tr(bt + k0 * ldb, ldb));
}
template <typename T, int K>
__device__ __forceinline__ void tile_mma_bt(f32x4& acc, const T* a, int lda, const T* b, int ldb) {
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += 32) mma(acc, ld_frag(a + k0, lda), ld_frag_tr(b + k0 * ldb, ldb));
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

template <typename T> __device__ __forceinline__ T to(float x) { return static_cast<T>(x); }
template <typename T> __device__ __forceinline__ float f32(T x) { return static_cast<float>(x); }

// Split x into a bf16 head and a bf16 tail with x ~= head + tail to about
// 2^-17 relative; used where an fp32 operand has to enter a bf16 product
// without losing the precision the covariance correction needs.
__device__ __forceinline__ void split_bf16(float x, bf16_t& hi, bf16_t& lo) {
  hi = static_cast<bf16_t>(x);
  lo = static_cast<bf16_t>(x - static_cast<float>(hi));
}

// Sum over the 16 lanes that share l / 16 (the lanes holding one tile row).
__device__ __forceinline__ float row16_sum(float x) {
  x += __shfl_xor(x, 1);
  x += __shfl_xor(x, 2);
  x += __shfl_xor(x, 4);
  x += __shfl_xor(x, 8);
  return x;
}

// Blocks are dealt to the 8 XCDs round-robin by linear id.  Renumber so that
// consecutive logical ids (the tiles of one head, which read the same q/k
// chunks) sit on one XCD and share its L2.
__device__ __forceinline__ int xcd_logical_block(int x, int nblocks) {
  if (nblocks % 8 != 0) return x;
  return (x % 8) * (nblocks / 8) + x / 8;
}

// Row offset of token (b, t, h) in a [B, T, H, D] tensor, in elements.
__device__ __forceinline__ size_t tok_off(int b, int t, int h, int T, int H, int D) {
  return (((size_t)b * T + t) * H + h) * (size_t)D;
}

// One 64-row chunk of a [*, D] token tensor held in registers as vectors of 8
// elements (16 bytes for bf16, 32 for fp32), so tiles of either dtype share
// one lane -> element mapping: lane l of every wave owns row l, wave w owns
// column groups w, w+4, ...  With the row in the lane index, a transposed LDS
// store (D rows, chunk index contiguous) writes 64 consecutive elements per
// instruction and is free of bank conflicts.  Rows >= n are zero.  Loads are
// branch-free (clamped row, then select), so a whole tile is in flight at
// once and can be issued a chunk ahead of its use.
template <typename T, int D, int NT = kThreads>
struct ChunkTile {
  static constexpr int VE = 8;
  static constexpr int NW = NT / 64;  // waves sharing the tile
  static constexpr int NV = kChunk * D / VE / NT;
  static_assert(NV >= 1 && kChunk * D % (VE * NT) == 0, "tile split");
  typedef T vec_t __attribute__((ext_vector_type(VE)));
  vec_t v[NV];
  bool ok;  // this lane's row lies inside the sequence

  __device__ __forceinline__ static int row() { return threadIdx.x & 63; }
  __device__ __forceinline__ static int col(int u) { return ((threadIdx.x >> 6) + NW * u) * VE; }

  // Issue the loads of rows [0, n) of the chunk at src (row pitch gstride
  // elements), n >= 1.  Rows >= n read row n-1 and are zeroed at use, so
  // nothing here waits for the data.
  __device__ __forceinline__ void load(const T* src, size_t gstride, int n) {
    const int r = row();
    ok = r < n;
    const T* p = src + (size_t)(ok ? r : n - 1) * gstride;
#pragma unroll
    for (int u = 0; u < NV; ++u) v[u] = *reinterpret_cast<const vec_t*>(p + col(u));
  }
  __device__ __forceinline__ vec_t get(int u) const {
    vec_t z;
#pragma unroll
    for (int e = 0; e < VE; ++e) z[e] = static_cast<T>(0.f);
    return ok ? v[u] : z;
  }
  __device__ __forceinline__ void store(T* dst, int ld) const {
#pragma unroll
    for (int u = 0; u < NV; ++u) *reinterpret_cast<vec_t*>(dst + row() * ld + col(u)) = get(u);
  }
  template <typename U>
  __device__ __forceinline__ void store_t(U* dstT, int ldT) const {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const vec_t x = get(u);
#pragma unroll
      for (int e = 0; e < VE; ++e) dstT[(col(u) + e) * ldT + row()] = static_cast<U>(static_cast<float>(x[e]));
    }
  }
  // fp32 copy, row-major; an odd pitch keeps it conflict-free for lane = row
  __device__ __forceinline__ void store_f32(float* dst, int ld) const {
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const vec_t x = get(u);
#pragma unroll
      for (int e = 0; e < VE; ++e) dst[row() * ld + col(u) + e] = static_cast<float>(x[e]);
    }
  }
};

// x, opaque to the optimiser: addresses derived from it are formed where they
// are used instead of being hoisted out of a loop and held in registers.
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// One 64-row chunk of a [*, D] token tensor staged for a row-major LDS copy,
// with coalesced global loads: vector e = tid + NT u (8 elements) is row
// e / (D / 8), column 8 (e % (D / 8)), so consecutive lanes read consecutive
// 16- or 32-byte pieces of a row and one wave instruction covers whole rows.
// Rows >= n read row n - 1 and are zeroed at use, so issuing the loads never
// waits for data.  With kWhole, a tile whose rows all lie inside the sequence
// (n >= 64, uniform over the workgroup) takes a branch without the clamping
// and the masks (fewer vector instructions per chunk in a loop over chunks;
// in a kernel that stages one chunk the branch only adds code).
template <typename T, int D, int NT = kThreads, bool kWhole = false>
struct RowTile {
  static constexpr int VE = 8;
  static constexpr int VPR = D / VE;                  // vectors per row
  static constexpr int TOT = kChunk * VPR;            // vectors in the tile
  static constexpr int NV = (TOT + NT - 1) / NT;      // vectors per thread
  static_assert(D % VE == 0, "row split");
  typedef T elem_t;
  typedef T vec_t __attribute__((ext_vector_type(VE)));
  vec_t v[NV];
  uint32_t ok;  // bit u: vector u exists and its row lies inside the sequence
  bool full;    // kWhole: every row lies inside the sequence (uniform)

  __device__ __forceinline__ static bool mine(int u) { return TOT % NT == 0 || (int)threadIdx.x + NT * u < TOT; }
  __device__ __forceinline__ static int row(int u) { return ((int)threadIdx.x + NT * u) / VPR; }
  __device__ __forceinline__ static int col(int u) { return (((int)threadIdx.x + NT * u) % VPR) * VE; }

  __device__ __forceinline__ void load(const T* src, size_t gstride, int n) {
    ok = 0;
    full = kWhole && n >= kChunk;
    if (full) {  // whole chunk: no clamping (the row offsets do not depend on n)
#pragma unroll
      for (int u = 0; u < NV; ++u)
        if (mine(u)) v[u] = *reinterpret_cast<const vec_t*>(src + (size_t)row(u) * gstride + col(u));
      return;
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      if (!mine(u)) continue;
      const int r = row(u);
      ok |= (r < n ? 1u : 0u) << u;
      v[u] = *reinterpret_cast<const vec_t*>(src + (size_t)(r < n ? r : n - 1) * gstride + col(u));
    }
  }
  // load() with the thread index passed through opaque(): the row offsets are
  // formed at the loads instead of being hoisted out of a loop over chunks and
  // held in registers (for kernels short of registers)
  __device__ __forceinline__ void load_opaque(const T* src, size_t gstride, int n) {
    const int t = opaque((int)threadIdx.x);
    ok = 0;
    full = false;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      if (!(TOT % NT == 0 || t + NT * u < TOT)) continue;
      const int r = (t + NT * u) / VPR, c = ((t + NT * u) % VPR) * VE;
      ok |= (r < n ? 1u : 0u) << u;
      v[u] = *reinterpret_cast<const vec_t*>(src + (size_t)(r < n ? r : n - 1) * gstride + c);
    }
  }
  __device__ __forceinline__ vec_t get(int u) const {
    vec_t z;
#pragma unroll
    for (int e = 0; e < VE; ++e) z[e] = static_cast<T>(0.f);
    return (full || ((ok >> u) & 1u)) ? v[u] : z;
  }
  // fp32 copy, row-major (adjacent lanes write adjacent elements of a row)
  __device__ __forceinline__ void store_f32(float* dst, int ld) const {
#pragma unroll
    for (int u = 0; u < NV; ++u)
      if (mine(u)) {
        const vec_t x = get(u);
#pragma unroll
        for (int e = 0; e < VE; ++e) dst[row(u) * ld + col(u) + e] = static_cast<float>(x[e]);
      }
  }
  __device__ __forceinline__ void store(T* dst, int ld) const {
    if (full) {
#pragma unroll
      for (int u = 0; u < NV; ++u)
        if (mine(u)) *reinterpret_cast<vec_t*>(dst + row(u) * ld + col(u)) = v[u];
      return;
    }
#pragma unroll
    for (int u = 0; u < NV; ++u)
      if (mine(u)) *reinterpret_cast<vec_t*>(dst + row(u) * ld + col(u)) = get(u);
  }
};

// Per-row scale factors of a RowTile's vectors (a row's l2 normalisation
// 1 / |x|), loaded beside the tile so that their latency overlaps its own.
// `sc` points at the factor of the tile's row 0 and consecutive rows are
// `stride` apart; rows >= n repeat row n - 1, as the tile does.
template <typename Tile>
struct RowScales {
  float f[Tile::NV];
  __device__ __forceinline__ void load(const float* sc, size_t stride, int n) {
#pragma unroll
    for (int u = 0; u < Tile::NV; ++u)
      if (Tile::mine(u)) {
        const int r = Tile::row(u);
        f[u] = sc[(size_t)(r < n ? r : n - 1) * stride];
      }
  }
  __device__ __forceinline__ void apply(Tile& t) const {
#pragma unroll
    for (int u = 0; u < Tile::NV; ++u)
      if (Tile::mine(u))
#pragma unroll
        for (int e = 0; e < Tile::VE; ++e) t.v[u][e] = to<typename Tile::elem_t>(f32(t.v[u][e]) * f[u]);
  }
};

// One 64-row chunk of a [*, D] token tensor streamed from global memory
// straight into LDS (gfx950 global_load_lds_dwordx4: each lane's 16 bytes land
// at the wave's LDS base + 16 * lane), so a prefetch holds no registers.  The
// destination is row-major with pitch D (no padding); one wave instruction
// covers RPI whole rows, and the NW waves of the workgroup split the
// instructions.  Rows >= n repeat row n - 1; the caller masks them.  The data
// is visible to the workgroup after s_waitcnt vmcnt(0) and a barrier.
template <int D, int NW>
struct LdsStream {
  static constexpr int VPR = D * 2 / 16;   // 16-byte pieces per bf16 row
  static constexpr int RPI = 64 / VPR;     // rows per wave instruction
  static constexpr int NI = kChunk / RPI / NW;  // instructions per wave
  static_assert(VPR <= 64 && 64 % VPR == 0 && kChunk % (RPI * NW) == 0, "stream split");
  // instruction it (< NI) of this wave
  __device__ __forceinline__ static void load_one(const bf16_t* src, size_t gstride, int n, bf16_t* dst, int it) {
    typedef __attribute__((address_space(3))) void lds_void;
    const int l = lane_id(), w = wave_id();
    const int ins = w * NI + it;
    const int row = ins * RPI + l / VPR;
    const bf16_t* p = src + (size_t)(row < n ? row : n - 1) * gstride + (l % VPR) * 8;
    __builtin_amdgcn_global_load_lds((const void*)p, (lds_void*)(dst + ins * RPI * D), 16, 0, 0);
  }
  __device__ __forceinline__ static void load(const bf16_t* src, size_t gstride, int n, bf16_t* dst) {
#pragma unroll
    for (int it = 0; it < NI; ++it) load_one(src, gstride, n, dst, it);
  }
};

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup barrier that orders LDS only: waits for this wave's LDS
// operations, not for its global loads and stores (a __syncthreads() fence
// would also drain the vector-memory counter, i.e. every prefetch in flight).
// Also a compiler barrier for memory accesses.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Transposing LDS read (as ld_frag_tr) issued as inline assembly.  The
// compiler treats the builtin form as possibly reading data that a
// global_load_lds still in flight is writing and drains every outstanding
// vector-memory operation before it, which would serialise a streamed
// prefetch; this form is invisible to its counters, so the caller makes the
// result valid with lds_wait() before use (the LDS returns data in order, so
// the compiler's own waits for later reads stay correct).
__device__ __forceinline__ bf16x4 ds_read_tr16_asm(const void* p) {
  bf16x4 r;
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(a));
  return r;
}
// s_waitcnt lgkmcnt(0), with the fragments passed through it so that no use
// of them can be scheduled above the wait.
template <int N>
__device__ __forceinline__ void lds_wait(Frag<bf16_t> (&f)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(f[i].v));
}
// The same, leaving the K most recently issued LDS operations in flight.
template <int K, int N>
__device__ __forceinline__ void lds_wait_but(Frag<bf16_t> (&f)[N]) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(K) : "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(f[i].v));
}


// Fragment loads from a pointer that already includes the lane's offset.
// frag_at: 8 contiguous elements (ld_frag with p = tile + (l % 16) ld + 8 (l / 16)).
// frag_acc_at: elements 0..3 and 16..19 (ld_frag_acc with p = tile + (l % 16) ld + 4 (l / 16)).
// frag_tr_at: ld_frag_tr with p = base + (8 (l / 16) + (l % 16) / 4) ld + 4 (l % 4)
// for bf16, p = base + 8 (l / 16) ld + l % 16 for fp32.
template <typename T>
__device__ __forceinline__ Frag<T> frag_at(const T* p) {
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    f.v = *reinterpret_cast<const bf16x8*>(p);
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(p);
    f.hi = *reinterpret_cast<const f32x4*>(p + 4);
  }
  return f;
}
template <typename T>
__device__ __forceinline__ Frag<T> frag_acc_at(const T* p) {
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 16);
    f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  } else {
    f.lo = *reinterpret_cast<const f32x4*>(p);
    f.hi = *reinterpret_cast<const f32x4*>(p + 16);
  }
  return f;
}
template <typename T>
__device__ __forceinline__ Frag<T> frag_tr_at(const T* p, int ld) {
  Frag<T> f;
  if constexpr (sizeof(T) == 2) {
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * ld));
    f.v = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f.lo[e] = p[e * ld];
      f.hi[e] = p[(4 + e) * ld];
    }
  }
  return f;
}
template <typename T>
__device__ __forceinline__ int frag_tr_lane_off(int l, int ld) {
  const int g = l >> 4, j = l & 15;
  if constexpr (sizeof(T) == 2) return (8 * g + (j >> 2)) * ld + 4 * (j & 3);
  else return 8 * g * ld + j;
}
// As frag_tr_lane_off, with the 16 columns of the tile taken in pair order:
// fragment row m reads column 8 (m / 4) + m % 4 (columns 0..3, 8..11, 16..19,
// 24..27 of a 32-wide block; add 4 for the other half).  Two such tiles are
// the rows of a pair of accumulator tiles whose packed fragment has 8
// consecutive columns per lane group.
template <typename T>
__device__ __forceinline__ int frag_tr_pair_lane_off(int l, int ld) {
  const int g = l >> 4, j = l & 15;
  if constexpr (sizeof(T) == 2) return (8 * g + (j >> 2)) * ld + 8 * (j & 3);
  else return 8 * g * ld + 8 * (j >> 2) + (j & 3);
}

// Chunks of sequence b that hold tokens.  Without offsets, all N chunks of the
// [B, T] batch; with the offsets cu of a packed batch laid out padded (rows
// past each sequence's end zero), ceil(len_b / 64) with len_b = cu[b+1] - cu[b]
// clamped to [0, T]: the chunks past them hold only zero rows, which leave
// every state unchanged, so the state and output passes may skip them.
__device__ __forceinline__ int live_chunks(const int* cu, int b, int T, int N) {
  if (!cu) return N;
  int len = cu[b + 1] - cu[b];
  len = len < 0 ? 0 : (len > T ? T : len);
  return (len + kChunk - 1) / kChunk;
}

// Sequence b of a batch: its first row in the token tensors and its length.
// Without offsets (cu null) the batch is padded, [B, T, ...], and every
// sequence has T tokens; with offsets it is packed: sequence b is rows
// cu[b] .. cu[b + 1] - 1 of [rows, ...] tensors, its length cut at T.
struct Seq {
  long long row0;
  int len;
};
__device__ __forceinline__ Seq seq_of(const int* cu, int b, int T) {
  if (!cu) return Seq{(long long)b * T, T};
  int len = cu[b + 1] - cu[b];
  len = len < 0 ? 0 : (len > T ? T : len);
  return Seq{(long long)cu[b], len};
}
// Offset of token t of sequence q, head h, in a [rows, H, D] tensor (elements).
__device__ __forceinline__ size_t seq_off(const Seq& q, int t, int h, int H, int D) {
  return ((size_t)(q.row0 + t) * H + h) * (size_t)D;
}
// Index of token t of sequence q, head h, in a [rows, H] tensor.
__device__ __forceinline__ size_t seq_idx(const Seq& q, int t, int h, int H) {
  return (size_t)(q.row0 + t) * H + h;
}

// Sum over aligned groups of n consecutive lanes (n = 2, 4, 8, 16), by
// swizzles (no address registers).
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16, "group");
  x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x041F));
  if constexpr (N >= 4) x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x081F));
  if constexpr (N >= 8) x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x101F));
  if constexpr (N >= 16) x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x201F));
  return x;
}

// Scalar per-token value prefetched by lane `row` (clamped address, zeroed at use).
struct RowScalar {
  float x;
  bool ok;
  __device__ __forceinline__ void load(const float* p, size_t stride, int row, int n) {
    ok = row < n;
    x = p[(size_t)(ok ? row : n - 1) * stride];
  }
  __device__ __forceinline__ float get() const { return ok ? x : 0.f; }
};

}  // namespace ccq
