// ccq_kernels.h -- internal launch interface between the C ABI (ccq_api.cpp)
// and the HIP kernel files.  Not installed; not part of the ABI.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ccq {

// Query contraction (Eq. clean evaluated chunkwise, App. B / Alg. 1).
struct CleanArgs {
  const void* q;      // [B,T,H,dk] io
  const void* k;      // [B,T,H,dk] io
  const float* lam;   // [B,T,H]
  const float* C0;    // [B,H,dk,dk] or null
  const float* mu0;   // [B,H,dk] or null
  void* qclean;       // [B,T,H,dk] io (workspace)
  float* qclean_dbg;  // [B,T,H,dk] fp32 or null
  float* CT;          // [B,H,dk,dk] or null
  float* muT;         // [B,H,dk] or null
  int B, T, H, dk;
  int centered;
  int64_t t0;
};

// GLA chunk forward reading the cleaned queries.
struct GlaArgs {
  const void* qc;     // [B,T,H,dk] io (cleaned queries)
  const void* k;      // [B,T,H,dk] io
  const void* v;      // [B,T,H,dv] io
  const void* g;      // [B,T,H,dk] gate dtype
  const float* S0;    // [B,H,dv,dk] or null
  void* o;            // [B,T,H,dv] io
  float* ST;          // [B,H,dv,dk] or null
  int B, T, H, dk, dv;
  float scale;
};

// Gated DeltaNet WY/UT chunk transform (chunk-parallel).
struct WyArgs {
  const void* k;         // [B,T,H,dk] io
  const void* v;         // [B,T,H,dv] io
  const float* logalpha; // [B,T,H]
  const float* beta;     // [B,T,H]
  void* W;               // [B*H, N, C, dk] io (workspace)
  float* Ut;             // [B*H, N, C, dv] fp32 (workspace)
  int B, T, H, dk, dv;
};

// Gated DeltaNet chunk forward (sequential over chunks).
struct GdnArgs {
  const void* qc;        // [B,T,H,dk] io (cleaned queries)
  const void* k;         // [B,T,H,dk] io
  const float* logalpha; // [B,T,H]
  const void* W;         // workspace, as WyArgs
  const float* Ut;       // workspace, as WyArgs
  const float* S0;       // [B,H,dv,dk] or null
  void* o;               // [B,T,H,dv] io
  float* ST;             // [B,H,dv,dk] or null
  int B, T, H, dk, dv;
  float scale;
};

// Each launcher returns hipSuccess or the launch error.  is_bf16 selects the
// io dtype (bf16 or fp32); shapes are validated by the caller.
hipError_t launch_clean(const CleanArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gla_fwd(const GlaArgs& a, bool is_bf16, bool gate_bf16, hipStream_t st);
hipError_t launch_gdn_wy(const WyArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_gdn_fwd(const GdnArgs& a, bool is_bf16, hipStream_t st);
hipError_t launch_copy_or_zero(float* dst, const float* src, size_t n, hipStream_t st);

// Supported-shape predicates (used by validation before any launch).
bool clean_supported(int dk, bool is_bf16);
bool gla_supported(int dk, int dv, bool is_bf16);
bool gdn_supported(int dk, int dv, bool is_bf16);

}  // namespace ccq
