// ccq_kernels.h -- internal launch interface between the C ABI (ccq_api.cpp)
// and the HIP kernel files.  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ccq {

// Query contraction (Eq. clean evaluated chunkwise, App. B / Alg. 1):
// out = base - lam * Sigma_t x  (base = x when null).  The backward pass runs
// the output kernel again on x = dL/dq_clean, since (I - lam Sigma)^T =
// I - lam Sigma, reusing the key statistics of the forward.
//
// The sequence is cut into segments of `seg` chunks.  Key statistics are
// formed per segment (clean_gram, clean_prefix); each segment's outputs then
// need only its entry statistics and its own keys (clean_out walks the
// segment's chunks in order), so the segments run in parallel.
//
// dk x dk statistics are stored fragment-native, in the order a 16x16 MFMA
// accumulator keeps them: element (m, n), the coefficient of x_m in (C x)_n,
// sits in tile (n / 16) (dk / 16) + m / 16 (1 KB fp32 per tile), lane
// n % 16 + 16 ((m % 16) / 4), slot m % 4.
struct CleanArgs {
  const void* q;      // x: [B,T,H,dk] io
  const void* k;      // [B,T,H,dk] io
  const float* lam;   // [B,T,H]
  const float* C0;    // [B,H,dk,dk] or null
  const float* mu0;   // [B,H,dk] or null
  void* qclean;       // out: [B,T,H,dk] io
  float* qclean_dbg;  // out in fp32, or null
  float* CT;          // [B,H,dk,dk] or null
  float* muT;         // [B,H,dk] or null
  const float* base;  // [B,T,H,dk] fp32 or null
  float* corr;        // Sigma_t x_t, [B,T,H,dk] fp32, or null
  float* mdot;        // m_t . x_t (raw key sum), [B,T,H] fp32, or null
  // workspace: NC = chunks, NS = segments per sequence
  float* gram;        // [B*H, NS, dk*dk] raw segment sums of k k^T, fragment-native
  void* sprime;       // [B*H, NS, dk*dk] io: entry second moment about c_s,
                      // fragment-native
  float* csum;        // [B*H, NC, dk] key sum of every chunk
  float* ssum;        // [B*H, NS, dk] key sum of every segment
  int B, T, H, dk;
  int centered;
  int seg;            // chunks per segment
  int64_t t0;
  // packed batch: sequence b is rows cu[b] .. cu[b+1] - 1 of [rows, H, d] token
  // tensors (length cut at T), or null for a padded [B, T, H, d] batch; the
  // workspace keeps its padded per-chunk layout either way
  const int* cu = nullptr;
  // raw q, k with per-row l2 normalisation folded in: token t, head h is scaled
  // by rq / rk [rows, H] fp32 (1 / max(|x|, eps)) as it is staged, or null
  const float* rq = nullptr;
  const float* rk = nullptr;
  // decay-aligned statistics (Gated DeltaNet): the per-token log decays
  // [rows, H] fp32, or null for the undecayed statistics of the paper; every
  // sum above is then weighted by the decay from the key to the point it is
  // taken at (the end of a chunk or segment) and token counts become the
  // decayed counts
  const float* la = nullptr;
  float* sdec = nullptr;  // [B*H, NS, 2] workspace: each segment's weight sum and decay
};

// GLA state recurrence (sequential over chunks) for one 64-channel tile of S.
// The chunks are cut into segments of `seg` (0: one segment); every segment
// starts from zero (the first from S0), so the segments run in parallel, and
// its chunk-entry states are the contributions of its own earlier chunks.
// With one segment they are the chunk-entry states S_r themselves.  Because
// the GLA transition is diagonal, the true S_r is the local state plus the
// segment's entry state scaled per key channel by the decay since the
// segment began (cdec); gla_scan forms the entry states from the segment
// totals (segsum, segdec).
struct GlaStateArgs {
  const void* k;      // [B,T,H,dk] io
  const void* v;      // [B,T,H,dv] io
  const void* g;      // [B,T,H,dk] gate dtype
  const float* S0;    // [B,H,dv,dk] or null
  float* ST;          // [B,H,dv,dk] or null (one segment only)
  void* states;       // [B*H, N, dv, dk] io: chunk-entry local states
  int B, T, H, dk, dv;
  int seg;            // chunks per segment, 0 = all
  float* segsum;      // [B*H, NS, dv, dk] fp32: local state at each segment's end (NS > 1)
  float* segdec;      // [B*H, NS, dk] fp32: e^{sum of the segment's log decays}
  float* cdec;        // [B*H, N, dk] fp32: e^{log decays of the segment before each chunk}
  float scale;        // read scale (the reverse scan of the training step only)
  const int* cu = nullptr;  // packed-batch offsets (device), as CleanArgs
  const float* rk = nullptr;  // key row scales, as CleanArgs
  int group = 1;  // forward: S_r stored for every group-th chunk only (the output groups)
};

// Entry state of every segment, E_0 = 0 (S0 is inside segment 0's states),
// E_{j+1} = E_j diag(segdec_j) + segsum_j; the last one gives S_T.
struct GlaScanArgs {
  const float* segsum;
  const float* segdec;
  void* entries;      // [B*H, NS, dv, dk] io (segment 0 unused)
  float* ST;          // [B,H,dv,dk] or null
  int B, H, dk, dv, NS;
};

// GLA output, one workgroup per (chunk, 64-wide value slice).
struct GlaOutArgs {
  const void* qc;     // [B,T,H,dk] io (cleaned queries)
  const void* k;      // [B,T,H,dk] io
  const void* v;      // [B,T,H,dv] io
  const void* g;      // [B,T,H,dk] gate dtype
  const void* states; // [B*H, N, dv, dk] io
  void* o;            // [B,T,H,dv] io
  int B, T, H, dk, dv;
  float scale;
  int seg;              // chunks per segment of the state pass (0 = one segment)
  const void* entries;  // [B*H, NS, dv, dk] io, or null with one segment
  const float* cdec;    // [B*H, N, dk] fp32, or null with one segment
  const int* cu = nullptr;  // packed-batch offsets (device), as CleanArgs
  const float* rk = nullptr;  // key row scales, as CleanArgs
  int group = 1;  // chunks per workgroup, S carried between them (gla_out_group)
};

// Gated DeltaNet chunk transform (chunk-parallel): Tm = (I + A)^{-1} and the
// chunk's decay coefficients.
struct TriArgs {
  const void* k;         // [B,T,H,dk] io
  const float* logalpha; // [B,T,H]
  const float* beta;     // [B,T,H]
  void* Tm;              // [B*H, N, C, C] io (workspace), columns in acc_pos order
  float* gam;            // [B*H, N, 5, C] fp32 (workspace): gamma_j (cumulative log
                         // decay in the chunk), beta_j e^{gamma_j}, beta_j,
                         // e^{gamma_C - gamma_j}, e^{gamma_C}
  int B, T, H, dk, dv;
  const int* cu = nullptr;  // packed-batch offsets [B+1] (device), as CleanArgs, or null
  // key row scales, as CleanArgs: the keys of A are scaled as staged, and the
  // coefficients beta e^gamma and e^{gamma_C - gamma} that multiply key rows
  // in the state pass and the output kernel's carry are stored times rk
  const float* rk = nullptr;
};

// Gated DeltaNet state recurrence (sequential over chunks): writes the
// chunk-entry states S_r and the corrected values U of every chunk.
struct GdnArgs {
  const void* k;         // [B,T,H,dk] io
  const void* v;         // [B,T,H,dv] io
  const float* beta;     // [B,T,H]
  const void* Tm;        // workspace, as TriArgs
  const float* gam;      // workspace, as TriArgs
  const float* S0;       // [B,H,dv,dk] or null
  float* ST;             // [B,H,dv,dk] or null
  void* states;          // [B*H, N, dv/16, dk/32, 16, 32] io (workspace): S_r
                         // (fragment-native, rows in natural feature order),
                         // stored for chunks r with r % sstride == 0
  void* U;               // [B*H, N, dv/16, 2, 16, 32] io (workspace): U^T, rows in
                         // acc_pos order (fragment-native), every chunk
  int B, T, H, dk, dv;
  int sstride = 1;
  const int* cu = nullptr;  // as TriArgs
};

// Gated DeltaNet output, one workgroup per group of `group` chunks (the
// state pass stored S_r for the first chunk of every group: sstride = group).
struct GdnOutArgs {
  const void* qc;        // [B,T,H,dk] io (cleaned queries)
  const void* k;         // [B,T,H,dk] io
  const float* gam;      // workspace, as TriArgs
  const void* states;    // as GdnArgs
  const void* U;         // as GdnArgs
  void* o;               // [B,T,H,dv] io
  int B, T, H, dk, dv;
  float scale;
  int group = 1;
  const int* cu = nullptr;  // as TriArgs
  const float* rk = nullptr;  // key row scales (the scores'; the carry's come with the coefficients)
};

// ---- training step (CCQ-GLA backward) ----
// Reverse scan of the state adjoint dS (decayed like S); stores the adjoint
// of the state leaving each chunk.
struct DstateArgs {
  const void* qc;     // [B,T,H,dk] io (cleaned queries)
  const void* g;      // [B,T,H,dk] gate dtype
  const void* dO;     // [B,T,H,dv] io
  void* dstates;      // [B*H, N, dv, dk] io
  int B, T, H, dk, dv;
  float scale;
};

// Chunk-parallel GLA gradients given S_r and dS_{r+1}.
struct GlaBwdArgs {
  const void* qc; const void* k; const void* v; const void* g; const void* dO;
  const void* states;   // [B*H, N, dv, dk] io
  const void* dstates;  // [B*H, N, dv, dk] io
  const float* corr;    // Sigma_t q_t, [B,T,H,dk] fp32
  float* dqc;           // dL/dq_clean [B,T,H,dk] fp32
  void* dqc_io;         // same, io dtype
  float* dk_gla;        // GLA part of dL/dk [B,T,H,dk] fp32
  void* dv_out;         // [B,T,H,dv] io
  float* db;            // dL/d(cumulative log decay) [B,T,H,dk] fp32
  float* dg_next;       // decay gradient at the first token of the next chunk [B*H, N, dk]
  float* dlam;          // [B,T,H]
  int B, T, H, dk, dv;
  float scale;
};

// dg_s = sum_{t >= s} db_t: the chunk's own rows plus dg_next.
struct DgArgs {
  const float* db;
  const float* dg_next;
  void* dg;             // [B,T,H,dk] gate dtype
  int B, T, H, dk;
};

// Key gradient of the contraction (suffix sums of an undecayed dk x dk state,
// formed per segment of chunks, then a reverse walk inside every segment).
struct CcqDkArgs {
  const void* q;        // [B,T,H,dk] io
  const void* k;        // [B,T,H,dk] io
  const void* u;        // dL/dq_clean, io
  const float* lam;     // [B,T,H]
  const float* mdot_q;  // m_t . q_t
  const float* mdot_u;  // m_t . u_t
  const float* dk_gla;  // [B,T,H,dk] fp32, added to the result
  void* dk_out;         // [B,T,H,dk] io
  int B, T, H, dk;
  int centered;
  int seg;              // chunks per segment (NS = ceil(N / seg) segments)
  float* hseg;          // [B*H, NS, dk, dk] fp32 workspace: each segment's H
  float* dseg;          // [B*H, NS, dk] fp32 workspace: each segment's D
  float* dchunk;        // [B*H, N, dk] fp32 workspace: each chunk's D
};

// ---- training step (CCQ-Gated DeltaNet backward) ----
// Per chunk, with the forward's Tm = (I + A)^{-1}: the decayed causal scores
// transposed, PT[j][i] = e^{gamma_i - gamma_j} (qc_i . k_j) for j <= i (else 0),
// plain row-major, and Tm^T with every row in acc_pos order.
struct GdnPrepArgs {
  const void* qc;        // [B,T,H,dk] io (cleaned queries)
  const void* k;         // [B,T,H,dk] io
  const float* gam;      // forward workspace, as TriArgs
  const void* Tm;        // forward workspace, as TriArgs
  void* PT;              // [B*H, N, C, C] io
  void* TmT;             // [B*H, N, C, C] io
  int B, T, H, dk, dv;
};

// Reverse scan of the state adjoint D = dS_{r+1} over the chunks of one head:
//   dU = PT (s dO) + diag(e^{gamma_C - gamma}) K D^T,   dR = Tm^T dU,
//   D <- e^{gamma_C} D + (s dO)^T diag(e^gamma) Qc - dR^T diag(beta e^gamma) K.
// Stores D (the adjoint of the state leaving each chunk) and dR.
struct GdnDstateArgs {
  const void* qc; const void* k; const void* dO;
  const float* gam;      // forward workspace, as TriArgs
  const void* PT;        // as GdnPrepArgs
  const void* TmT;       // as GdnPrepArgs
  void* dstates;         // [B*H, N, dv, dk] io, plain row-major
  void* dR;              // [B,T,H,dv] io
  int B, T, H, dk, dv;
  float scale;
};

// Chunk-parallel Gated DeltaNet gradients given S_r, U, dS_{r+1} and dR.
struct GdnBwdArgs {
  const void* qc; const void* k; const void* v; const void* dO;
  const float* gam;      // forward workspace, as TriArgs
  const void* states;    // forward workspace S_r, as GdnArgs (fragment-native)
  const void* U;         // forward workspace U^T, as GdnArgs (fragment-native)
  const void* dstates;   // as GdnDstateArgs
  const void* dR;        // as GdnDstateArgs
  const float* corr;     // Sigma_t q_t, [B,T,H,dk] fp32
  float* dqc;            // dL/dq_clean [B,T,H,dk] fp32
  void* dqc_io;          // same, io dtype
  float* dk_bb;          // backbone part of dL/dk [B,T,H,dk] fp32
  void* dv_out;          // [B,T,H,dv] io
  float* dlogalpha;      // [B,T,H]
  float* dbeta;          // [B,T,H]
  float* dlam;           // [B,T,H]
  int B, T, H, dk, dv;
  float scale;
};

// ---- recurrent decode (one token per sequence, cache updated in place) ----
struct DecodeArgs {
  const void* q;         // [B,H,dk] io
  const void* k;         // [B,H,dk] io
  const void* v;         // [B,H,dv] io
  const void* g;         // GLA: [B,H,dk] gate dtype; Gated DeltaNet: [B,H] fp32 log alpha
  const float* beta;     // Gated DeltaNet: [B,H] fp32
  const float* lam;      // [B,H] fp32
  float* S;              // [B,H,dv,dk] fp32, in place
  float* C;              // [B,H,dk,dk] fp32 (Cbar), in place
  float* mu;             // [B,H,dk] fp32, in place
  float* cq;             // [B,H,dk] fp32 workspace: Cbar_t q (split step only)
  void* o;               // [B,H,dv] io
  int B, H, dk, dv;
  int centered;
  float scale;
  int64_t t0;            // tokens before this one (its position is t0 + 1)
};

// ---- pre-processing: per-head l2 normalisation and the gate ----
constexpr int kPrepMaxHeads = 16;
constexpr size_t kPrepMaxLds = 65536;  // W_lambda staged in LDS (fp32)
struct PrepArgs {
  const void* q_raw;     // [B,T,H,dk] io
  const void* k_raw;     // [B,T,H,dk] io
  const float* w;        // [H, H*dk] fp32
  const float* b;        // [H] fp32
  void* q;               // [B,T,H,dk] io (may be q_raw), or null with rq
  void* k;               // [B,T,H,dk] io (may be k_raw), or null with rk
  float* lam;            // [B,T,H] fp32
  int B, T, H, dk;
  // instead of the normalised rows: the row scales 1 / max(|x|, 1e-12) [B,T,H]
  float* rq = nullptr;
  float* rk = nullptr;
};

// Each launcher returns hipSuccess or the launch error.  is_bf16 selects the
// io dtype (bf16 or fp32); shapes are validated by the caller.
hipError_t launch_clean_gram(const CleanArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_clean_prefix(const CleanArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_clean_out(const CleanArgs& a, bool is_bf16, hipStream_t st);
// Chunks per segment of the query contraction for bh heads of nc chunks.  Each
// segment is one workgroup walking its chunks in order, one workgroup per
// compute unit at a time, so the pass takes about (rounds of 256 workgroups) x
// (chunks per segment) chunk steps: the segment length (2 to 64) that
// minimises that, the longest on a tie (fewer segment statistics).
inline int clean_seg(long long bh, long long nc) {
  int best = 2;
  long long best_cost = -1;
  for (int seg = 2; seg <= 64; ++seg) {
    const long long wgs = bh * ((nc + seg - 1) / seg);
    const long long cost = ((wgs + 255) / 256) * (seg < nc ? seg : nc);
    if (best_cost < 0 || cost <= best_cost) {
      best_cost = cost;
      best = seg;
    }
  }
  return best;
}
hipError_t launch_gla_state(const GlaStateArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st);
hipError_t launch_gla_out(const GlaOutArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st);
hipError_t launch_gla_scan(const GlaScanArgs& a, bool is_bf16, hipStream_t st);
// Chunks per segment of the GLA state pass (0: one segment) for bh heads of
// nc chunks.  A workgroup carries one 64 x (16 NVT) tile of S through its
// segment's chunks, two workgroups per compute unit; the segments then meet
// in a scan.  The segment count minimises rounds of 512 workgroups x chunks
// per segment, plus two chunk steps for the scan when there is more than one
// segment (of at least 4 chunks); the fewest segments on a tie.
inline int gla_seg(long long bh, long long nc, int dk, int dv) {
  const long long tiles = bh * (dk / 64) * (dv / 64);
  long long best_ns = 1, best_cost = -1;
  for (long long ns = 1; ns <= 64 && ns <= nc; ++ns) {
    const long long sl = (nc + ns - 1) / ns;
    if ((nc + sl - 1) / sl != ns || (ns > 1 && sl < 4)) continue;  // ns segments of sl >= 4 chunks
    const long long cost = ((tiles * ns + 511) / 512) * sl + (ns > 1 ? 2 : 0);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best_ns = ns;
    }
  }
  return best_ns > 1 ? (int)((nc + best_ns - 1) / best_ns) : 0;
}
hipError_t launch_gdn_tri(const TriArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gdn_state(const GdnArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gdn_out(const GdnOutArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_copy_or_zero(float* dst, const float* src, size_t n, hipStream_t st);

hipError_t launch_gla_dstate(const DstateArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st);
hipError_t launch_gla_bwd_chunk(const GlaBwdArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st);
hipError_t launch_gla_dg(const DgArgs& a, bool gate_bf16, hipStream_t st);
hipError_t launch_ccq_dk(const CcqDkArgs& a, bool is_bf16, hipStream_t st);
// Training-step shapes: bf16 dk in {64, 128} (and 256 for Gated DeltaNet), fp32 dk = 64.
bool bwd_supported(int dk, int dv, bool is_bf16, bool gdn);
hipError_t launch_gdn_bwd_prep(const GdnPrepArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gdn_dstate(const GdnDstateArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gdn_bwd_chunk(const GdnBwdArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_decode(const DecodeArgs& a, bool gdn, bool is_bf16, bool gate_bf16, hipStream_t st);
bool decode_supported(int dk, int dv);
bool decode_split(long long bh, int dk, int dv);  // two launches over 16-row blocks (needs the workspace)
hipError_t launch_prep(const PrepArgs& a, bool is_bf16, hipStream_t st);
bool prep_supported(int H, int dk);

// Packed batches: rows of sequence b are cu[b] .. cu[b+1] - 1 of a [rows, ...]
// tensor whose rows are row_bytes wide (a multiple of 4).  to_padded: packed
// -> [B, T, ...] with the rows past each sequence's end zeroed; else the
// sequences' rows back from padded to packed.
hipError_t launch_varlen_copy(void* dst, const void* src, const int* cu, int B, int T, size_t row_bytes,
                              bool to_padded, hipStream_t st);

// Supported-shape predicates (used by validation before any launch).
bool clean_supported(int dk, bool is_bf16);
bool gla_supported(int dk, int dv, bool is_bf16);
// Chunks per output workgroup of the GLA forward (1: one chunk each).
int gla_out_group(int B, int H, int T, int dk, int dv, bool is_bf16);
bool gdn_supported(int dk, int dv, bool is_bf16);
// Chunks per output workgroup (and state stride) for a forward pass.
int gdn_out_group(int B, int H, int T, int dk, int dv, bool is_bf16);
// Whether the output kernel can carry S through a group at this shape.
bool gdn_out_carries(int dk, int dv, bool is_bf16);

}  // namespace ccq
