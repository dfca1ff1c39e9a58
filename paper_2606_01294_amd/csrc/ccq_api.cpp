// ccq_api.cpp -- the C ABI declared in include/ccq.h: argument validation,
// workspace layout and kernel dispatch.  Every check runs before the first
// launch, so an error return means nothing was enqueued.
#include "ccq.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "ccq_kernels.h"

// Scratch of the allocation-free forward (ccq_gdn_fwd_noalloc), one copy per
// device; see scratch_on_current_device below.
static constexpr size_t kScratchBytes = CCQ_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// Per-host-thread kernel timing hook (ccq_trace_events).
struct Trace {
  hipEvent_t* ev = nullptr;
  int n = 0;
  int next = 0;
  bool nested = false;  // inside an entry point that wraps another one
};
thread_local Trace g_trace;

void trace_begin_call() {
  if (!g_trace.nested) g_trace.next = 0;
}
// An entry point built on another one numbers its own launches and the inner
// call's in one sequence.
struct TraceScope {
  TraceScope() {
    trace_begin_call();
    g_trace.nested = true;
  }
  ~TraceScope() { g_trace.nested = false; }
};

// Runs one launcher between the trace events of its slot, if tracing is on.
template <typename F>
hipError_t traced(hipStream_t st, F&& launch) {
  const int i = g_trace.next++;
  const bool on = g_trace.ev && 2 * i + 1 < g_trace.n;
  if (on && hipEventRecord(g_trace.ev[2 * i], st) != hipSuccess) return hipErrorUnknown;
  hipError_t e = launch();
  if (e == hipSuccess && on && hipEventRecord(g_trace.ev[2 * i + 1], st) != hipSuccess)
    return hipErrorUnknown;
  return e;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t esize(ccq_dtype d) { return d == CCQ_BF16 ? 2 : 4; }
bool dtype_ok(ccq_dtype d) { return d == CCQ_F32 || d == CCQ_BF16; }
bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Common shape checks.  Returns CCQ_OK or the error.
ccq_status check_shape(const ccq_shape* s, ccq_backbone bb) {
  if (!s) return CCQ_ERR_INVALID_ARG;
  if (s->B < 0 || s->T < 0 || s->H < 0 || s->t0 < 0) return CCQ_ERR_INVALID_ARG;
  if (!dtype_ok(s->io_dtype) || !dtype_ok(s->gate_dtype)) return CCQ_ERR_INVALID_ARG;
  if (s->centered != 0 && s->centered != 1) return CCQ_ERR_INVALID_ARG;
  if (s->decay_aligned != 0 && s->decay_aligned != 1) return CCQ_ERR_INVALID_ARG;
  if (bb != CCQ_GLA && bb != CCQ_GDN) return CCQ_ERR_INVALID_ARG;
  // the decay-aligned statistics: scalar decay (Gated DeltaNet), from empty statistics
  if (s->decay_aligned && (bb != CCQ_GDN || s->t0 != 0)) return CCQ_ERR_UNSUPPORTED;
  if (s->chunk != 64) return CCQ_ERR_UNSUPPORTED;
  const bool bf = s->io_dtype == CCQ_BF16;
  if (!ccq::clean_supported(s->dk, bf)) return CCQ_ERR_UNSUPPORTED;
  if (bb == CCQ_GLA ? !ccq::gla_supported(s->dk, s->dv, bf) : !ccq::gdn_supported(s->dk, s->dv, bf))
    return CCQ_ERR_UNSUPPORTED;
  // 32-bit grid and index headroom
  const long long ntok = (long long)s->B * s->T * s->H;
  if (ntok * (s->dk > s->dv ? s->dk : s->dv) > (1LL << 40)) return CCQ_ERR_UNSUPPORTED;
  if ((long long)s->B * s->H * ((s->T + 63) / 64) > (1LL << 30)) return CCQ_ERR_UNSUPPORTED;
  return CCQ_OK;
}

// Workspace of the query contraction: segment and chunk key statistics.
struct CleanWs {
  size_t gram = 0, sprime = 0, csum = 0, ssum = 0, sdec = 0;
};

template <typename Take>
CleanWs take_clean_ws(const ccq_shape* s, Take&& take) {
  const size_t bh = (size_t)s->B * s->H, dk = s->dk;
  const size_t nc = (s->T + 63) / 64, seg = ccq::clean_seg((long long)bh, (long long)nc);
  const size_t ns = (nc + seg - 1) / seg;
  CleanWs c;
  c.gram = take(bh * ns * dk * dk * 4);
  c.sprime = take(bh * ns * dk * dk * esize(s->io_dtype));
  c.csum = take(bh * nc * dk * 4);
  c.ssum = take(bh * ns * dk * 4);
  c.sdec = take(bh * ns * 2 * 4);  // decay-aligned statistics: segment weight sums and decays
  return c;
}

ccq::CleanArgs clean_args(const ccq_shape* s, char* ws, const CleanWs& c) {
  ccq::CleanArgs a{};
  a.gram = reinterpret_cast<float*>(ws + c.gram);
  a.sprime = ws + c.sprime;
  a.csum = reinterpret_cast<float*>(ws + c.csum);
  a.ssum = reinterpret_cast<float*>(ws + c.ssum);
  a.sdec = reinterpret_cast<float*>(ws + c.sdec);
  a.B = s->B;
  a.T = s->T;
  a.H = s->H;
  a.dk = s->dk;
  a.centered = s->centered;
  a.seg = ccq::clean_seg((long long)s->B * s->H, (s->T + 63) / 64);
  a.t0 = s->t0;
  return a;
}

// Key statistics of the contraction (depend on k only).
hipError_t run_clean_stats(const ccq::CleanArgs& a, bool bf, hipStream_t st) {
  hipError_t e = traced(st, [&] { return ccq::launch_clean_gram(a, bf, st); });
  if (e == hipSuccess) e = traced(st, [&] { return ccq::launch_clean_prefix(a, bf, st); });
  return e;
}

struct FwdLayout {
  size_t qclean = 0, states = 0, Tm = 0, gam = 0, U = 0, total = 0;
  size_t segsum = 0, segdec = 0, cdec = 0, entries = 0;  // GLA state pass in segments
  int gla_seg = 0;
  CleanWs clean;
};

// q_clean, the chunk-entry states S_r and, for Gated DeltaNet, the chunk
// transforms Tm, the cumulative log decays and the corrected values U.
FwdLayout fwd_layout(const ccq_shape* s, ccq_backbone bb) {
  FwdLayout L;
  const size_t ntok = (size_t)s->B * s->T * s->H;
  const size_t nchunk = (size_t)s->B * s->H * ((s->T + 63) / 64);
  const size_t e = esize(s->io_dtype);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align_up(bytes); return o; };
  L.qclean = take(ntok * s->dk * e);
  L.states = take(nchunk * s->dv * s->dk * e);
  L.clean = take_clean_ws(s, take);
  if (bb == CCQ_GLA) {
    const long long nc = (s->T + 63) / 64;
    L.gla_seg = ccq::gla_seg((long long)s->B * s->H, nc, s->dk, s->dv);
    if (L.gla_seg > 0) {
      const size_t bh = (size_t)s->B * s->H, ns = (nc + L.gla_seg - 1) / L.gla_seg;
      L.segsum = take(bh * ns * s->dv * s->dk * sizeof(float));
      L.segdec = take(bh * ns * s->dk * sizeof(float));
      L.cdec = take(nchunk * s->dk * sizeof(float));
      L.entries = take(bh * ns * s->dv * s->dk * e);
    }
  }
  if (bb == CCQ_GDN) {
    L.Tm = take(nchunk * 64 * 64 * e);
    L.gam = take(nchunk * 5 * 64 * sizeof(float));
    L.U = take(nchunk * 64 * s->dv * e);
  }
  L.total = off;
  return L;
}

// Suffix statistics of the contraction's key gradient (ccq_dk).
struct DkWs {
  size_t hseg = 0, dseg = 0, dchunk = 0;
};

template <typename Take>
DkWs take_dk_ws(const ccq_shape* s, Take&& take) {
  const size_t bh = (size_t)s->B * s->H, dk = s->dk;
  const size_t nc = (s->T + 63) / 64, seg = ccq::clean_seg((long long)bh, (long long)nc);
  const size_t ns = (nc + seg - 1) / seg;
  DkWs d;
  d.hseg = take(bh * ns * dk * dk * 4);
  d.dseg = take(bh * ns * dk * 4);
  d.dchunk = take(bh * nc * dk * 4);
  return d;
}

void set_dk_ws(ccq::CcqDkArgs& ka, const ccq_shape* s, char* ws, const DkWs& d) {
  ka.seg = ccq::clean_seg((long long)s->B * s->H, (s->T + 63) / 64);
  ka.hseg = reinterpret_cast<float*>(ws + d.hseg);
  ka.dseg = reinterpret_cast<float*>(ws + d.dseg);
  ka.dchunk = reinterpret_cast<float*>(ws + d.dchunk);
}

struct BwdLayout {
  size_t qclean, corr, mdq, mdu, states, dstates, dqc, dqc_io, dkg, db, dgn, total;
  CleanWs clean;
  DkWs dkws;
};

BwdLayout bwd_layout(const ccq_shape* s) {
  BwdLayout L{};
  const size_t ntok = (size_t)s->B * s->T * s->H;
  const size_t nchunk = (size_t)s->B * s->H * ((s->T + 63) / 64);
  const size_t e = esize(s->io_dtype);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align_up(bytes); return o; };
  L.qclean = take(ntok * s->dk * e);
  L.corr = take(ntok * s->dk * 4);
  L.mdq = take(ntok * 4);
  L.mdu = take(ntok * 4);
  L.states = take(nchunk * s->dv * s->dk * e);
  L.dstates = take(nchunk * s->dv * s->dk * e);
  L.dqc = take(ntok * s->dk * 4);
  L.dqc_io = take(ntok * s->dk * e);
  L.dkg = take(ntok * s->dk * 4);
  L.db = take(ntok * s->dk * 4);
  L.dgn = take(nchunk * s->dk * 4);  // dg at each next chunk's first token
  L.clean = take_clean_ws(s, take);
  L.dkws = take_dk_ws(s, take);
  L.total = off;
  return L;
}

// Training step of CCQ-Gated DeltaNet: the forward's q_clean, key statistics,
// chunk transforms, S_r and U, then the backward's PT, Tm^T, dS_{r+1} and dR.
struct GdnBwdLayout {
  size_t qclean, corr, mdq, mdu, states, Tm, gam, U, PT, TmT, dstates, dR, dqc, dqc_io, dkb, total;
  CleanWs clean;
  DkWs dkws;
};

GdnBwdLayout gdn_bwd_layout(const ccq_shape* s) {
  GdnBwdLayout L{};
  const size_t ntok = (size_t)s->B * s->T * s->H;
  const size_t nchunk = (size_t)s->B * s->H * ((s->T + 63) / 64);
  const size_t e = esize(s->io_dtype);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += align_up(bytes); return o; };
  L.qclean = take(ntok * s->dk * e);
  L.corr = take(ntok * s->dk * 4);
  L.mdq = take(ntok * 4);
  L.mdu = take(ntok * 4);
  L.states = take(nchunk * s->dv * s->dk * e);
  L.Tm = take(nchunk * 64 * 64 * e);
  L.gam = take(nchunk * 5 * 64 * sizeof(float));
  L.U = take(nchunk * 64 * s->dv * e);
  L.PT = take(nchunk * 64 * 64 * e);
  L.TmT = take(nchunk * 64 * 64 * e);
  L.dstates = take(nchunk * s->dv * s->dk * e);
  L.dR = take(ntok * s->dv * e);
  L.dqc = take(ntok * s->dk * 4);
  L.dqc_io = take(ntok * s->dk * e);
  L.dkb = take(ntok * s->dk * 4);
  L.clean = take_clean_ws(s, take);
  L.dkws = take_dk_ws(s, take);
  L.total = off;
  return L;
}

// T == 0: the final states are the initial ones (or zero).
ccq_status copy_initial_states(const ccq_shape* s, const float* S0, const float* C0,
                               const float* mu0, float* ST, float* CT, float* muT,
                               hipStream_t st) {
  const size_t bh = (size_t)s->B * s->H;
  hipError_t e = hipSuccess;
  if (ST && e == hipSuccess) e = ccq::launch_copy_or_zero(ST, S0, bh * s->dv * s->dk, st);
  if (CT && e == hipSuccess) e = ccq::launch_copy_or_zero(CT, C0, bh * s->dk * s->dk, st);
  if (muT && e == hipSuccess) e = ccq::launch_copy_or_zero(muT, mu0, bh * s->dk, st);
  return e == hipSuccess ? CCQ_OK : CCQ_ERR_HIP;
}

// Argument checks of the forward entry points (nothing is launched).
ccq_status check_forward_args(ccq_backbone bb, const ccq_shape* s, const void* q, const void* k,
                              const void* v, const void* g_or_la, const float* beta,
                              const float* lam, const float* S0, const float* C0,
                              const float* mu0, const void* o, const float* ST, const float* CT,
                              const float* muT, const float* q_clean_dbg, const void* workspace) {
  ccq_status rc = check_shape(s, bb);
  if (rc != CCQ_OK) return rc;
  if (s->decay_aligned && (C0 || mu0)) return CCQ_ERR_UNSUPPORTED;  // no cached W to continue from
  const size_t ntok = (size_t)s->B * s->T * s->H;
  const void* ptrs[] = {S0, C0, mu0, ST, CT, muT, q_clean_dbg, workspace};
  for (const void* p : ptrs)
    if (p && !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (ntok > 0) {
    const void* req[] = {q, k, v, g_or_la, lam, o};
    for (const void* p : req)
      if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
    if (bb == CCQ_GDN && (!beta || !aligned(beta))) return CCQ_ERR_INVALID_ARG;
  }
  return CCQ_OK;
}

// cu: device offsets of a packed batch (sequence b is rows cu[b] .. cu[b+1] - 1
// of the token tensors, cut at s->T), or null for a padded [B, T, ...] batch.
// Every kernel reads and writes the packed rows directly and walks only each
// sequence's own chunks; the workspace keeps its padded per-chunk layout.
ccq_status run_forward(ccq_backbone bb, const ccq_shape* s, const void* q, const void* k,
                       const void* v, const void* g_or_la, const float* beta, const float* lam,
                       const float* S0, const float* C0, const float* mu0, void* o, float* ST,
                       float* CT, float* muT, float* q_clean_dbg, void* workspace,
                       size_t ws_bytes, void* stream, const int32_t* cu = nullptr,
                       const float* rq = nullptr, const float* rk = nullptr) {
  ccq_status rc = check_forward_args(bb, s, q, k, v, g_or_la, beta, lam, S0, C0, mu0, o, ST, CT,
                                     muT, q_clean_dbg, workspace);
  if (rc != CCQ_OK) return rc;
  const FwdLayout L = fwd_layout(s, bb);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s->B == 0 || s->H == 0) return CCQ_OK;
  if (s->T == 0) return copy_initial_states(s, S0, C0, mu0, ST, CT, muT, st);
  if (!workspace || ws_bytes < L.total) return CCQ_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  const bool bf = s->io_dtype == CCQ_BF16;
  void* qclean = ws + L.qclean;
  const float* la = static_cast<const float*>(g_or_la);
  float* gam = reinterpret_cast<float*>(ws + L.gam);
  const bool gbf = s->gate_dtype == CCQ_BF16;
  trace_begin_call();
  // the backbone's chunk transforms (Gated DeltaNet) and state pass: chunk-entry
  // states S_r (and U)
  if (bb == CCQ_GDN) {
    ccq::TriArgs ta{k, la, beta, ws + L.Tm, gam, s->B, s->T, s->H, s->dk, s->dv};
    ta.cu = cu;
    ta.rk = rk;
    if (traced(st, [&] { return ccq::launch_gdn_tri(ta, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  }
  if (bb == CCQ_GLA) {
    // segments of the state pass run in parallel; a scan over the segment
    // totals gives every segment's entry state and S_T
    ccq::GlaStateArgs sa{k, v, g_or_la, S0, ST, ws + L.states, s->B, s->T, s->H, s->dk, s->dv};
    sa.cu = cu;
    sa.rk = rk;
    sa.group = ccq::gla_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);  // one state per output group
    if (L.gla_seg > 0) {
      sa.seg = L.gla_seg;
      sa.ST = nullptr;
      sa.segsum = reinterpret_cast<float*>(ws + L.segsum);
      sa.segdec = reinterpret_cast<float*>(ws + L.segdec);
      sa.cdec = reinterpret_cast<float*>(ws + L.cdec);
    }
    if (traced(st, [&] { return ccq::launch_gla_state(sa, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
    if (L.gla_seg > 0) {
      const int nc = (s->T + 63) / 64;
      ccq::GlaScanArgs ga{sa.segsum, sa.segdec, ws + L.entries, ST, s->B, s->H, s->dk, s->dv,
                          (nc + L.gla_seg - 1) / L.gla_seg};
      if (traced(st, [&] { return ccq::launch_gla_scan(ga, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
    }
  } else {
    ccq::GdnArgs da{k, v, beta, ws + L.Tm, gam, S0, ST, ws + L.states, ws + L.U, s->B, s->T, s->H,
                    s->dk, s->dv};
    da.sstride = ccq::gdn_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);  // one state per output group
    da.cu = cu;
    if (traced(st, [&] { return ccq::launch_gdn_state(da, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  }

  // the query contraction
  ccq::CleanArgs ca = clean_args(s, ws, L.clean);
  ca.q = q;
  ca.k = k;
  ca.lam = lam;
  ca.C0 = C0;
  ca.mu0 = mu0;
  ca.cu = cu;
  ca.rq = rq;
  ca.rk = rk;
  ca.qclean = qclean;
  ca.qclean_dbg = q_clean_dbg;
  ca.CT = CT;
  ca.muT = muT;
  if (s->decay_aligned) ca.la = la;  // keys weighted by the backbone's decay (check_shape: GDN)
  if (run_clean_stats(ca, bf, st) != hipSuccess) return CCQ_ERR_HIP;
  if (traced(st, [&] { return ccq::launch_clean_out(ca, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;

  // outputs from q_clean and the chunk-entry states
  if (bb == CCQ_GLA) {
    ccq::GlaOutArgs oa{qclean, k, v, g_or_la, ws + L.states, o, s->B, s->T, s->H, s->dk, s->dv, s->scale};
    oa.cu = cu;
    oa.rk = rk;
    oa.group = ccq::gla_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);  // as the state pass stored
    if (L.gla_seg > 0) {
      oa.seg = L.gla_seg;
      oa.entries = ws + L.entries;
      oa.cdec = reinterpret_cast<const float*>(ws + L.cdec);
    }
    if (traced(st, [&] { return ccq::launch_gla_out(oa, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  } else {
    ccq::GdnOutArgs oa{qclean, k, gam, ws + L.states, ws + L.U, o, s->B, s->T, s->H, s->dk, s->dv,
                       s->scale};
    oa.group = ccq::gdn_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);
    oa.cu = cu;
    oa.rk = rk;
    if (traced(st, [&] { return ccq::launch_gdn_out(oa, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  }
  return CCQ_OK;
}

// CCQ-Gated DeltaNet training step (arguments validated by the caller).
ccq_status gdn_fwd_bwd(const ccq_shape* s, const void* q, const void* k, const void* v,
                       const float* la, const float* beta, const float* lam, const void* dO,
                       void* o, void* dq, void* dk, void* dv, float* dla, float* dbeta,
                       float* dlam, void* workspace, size_t ws_bytes, void* stream) {
  const GdnBwdLayout L = gdn_bwd_layout(s);
  if (!workspace || ws_bytes < L.total) return CCQ_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const bool bf = s->io_dtype == CCQ_BF16;
  float* corr = reinterpret_cast<float*>(ws + L.corr);
  float* mdq = reinterpret_cast<float*>(ws + L.mdq);
  float* mdu = reinterpret_cast<float*>(ws + L.mdu);
  float* gam = reinterpret_cast<float*>(ws + L.gam);
  float* dqc = reinterpret_cast<float*>(ws + L.dqc);
  float* dkb = reinterpret_cast<float*>(ws + L.dkb);
  trace_begin_call();

  // forward: cleaned queries (with Sigma q and m.q kept), chunk transforms,
  // S_r and U, outputs
  ccq::CleanArgs c1 = clean_args(s, ws, L.clean);
  c1.q = q;
  c1.k = k;
  c1.lam = lam;
  c1.qclean = ws + L.qclean;
  c1.corr = corr;
  c1.mdot = mdq;
  if (run_clean_stats(c1, bf, st) != hipSuccess) return CCQ_ERR_HIP;
  if (traced(st, [&] { return ccq::launch_clean_out(c1, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::TriArgs ta{k, la, beta, ws + L.Tm, gam, s->B, s->T, s->H, s->dk, s->dv};
  if (traced(st, [&] { return ccq::launch_gdn_tri(ta, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GdnArgs sa{k, v, beta, ws + L.Tm, gam, nullptr, nullptr, ws + L.states, ws + L.U, s->B,
                  s->T, s->H, s->dk, s->dv};
  if (traced(st, [&] { return ccq::launch_gdn_state(sa, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GdnOutArgs oa{ws + L.qclean, k, gam, ws + L.states, ws + L.U, o, s->B, s->T, s->H, s->dk,
                     s->dv, s->scale};
  // every S_r is stored (the backward reads them); the output kernel still
  // reads only each group's first and carries S through the group
  oa.group = ccq::gdn_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);
  if (traced(st, [&] { return ccq::launch_gdn_out(oa, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  // backward: PT and Tm^T, the reverse state scan, chunk gradients, dq, dk
  ccq::GdnPrepArgs pa{ws + L.qclean, k, gam, ws + L.Tm, ws + L.PT, ws + L.TmT, s->B, s->T, s->H,
                      s->dk, s->dv};
  if (traced(st, [&] { return ccq::launch_gdn_bwd_prep(pa, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GdnDstateArgs da{ws + L.qclean, k, dO, gam, ws + L.PT, ws + L.TmT, ws + L.dstates, ws + L.dR,
                        s->B, s->T, s->H, s->dk, s->dv, s->scale};
  if (traced(st, [&] { return ccq::launch_gdn_dstate(da, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GdnBwdArgs ba{ws + L.qclean, k, v, dO, gam, ws + L.states, ws + L.U, ws + L.dstates,
                     ws + L.dR, corr, dqc, ws + L.dqc_io, dkb, dv, dla, dbeta, dlam, s->B, s->T,
                     s->H, s->dk, s->dv, s->scale};
  if (traced(st, [&] { return ccq::launch_gdn_bwd_chunk(ba, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::CleanArgs c2 = clean_args(s, ws, L.clean);  // same keys: statistics reused
  c2.q = ws + L.dqc_io;
  c2.k = k;
  c2.lam = lam;
  c2.qclean = dq;
  c2.base = dqc;
  c2.mdot = mdu;
  if (traced(st, [&] { return ccq::launch_clean_out(c2, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::CcqDkArgs ka{q, k, ws + L.dqc_io, lam, mdq, mdu, dkb, dk, s->B, s->T, s->H, s->dk,
                    s->centered};
  set_dk_ws(ka, s, ws, L.dkws);
  if (traced(st, [&] { return ccq::launch_ccq_dk(ka, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  return CCQ_OK;
}

// Padded copies of a packed batch, ahead of the padded path's own workspace.
struct VarlenLayout {
  size_t q = 0, k = 0, v = 0, gate = 0, beta = 0, lam = 0, o = 0;
  size_t dO = 0, dq = 0, dk = 0, dv = 0, dgate = 0, dbeta = 0, dlam = 0;
  size_t inner = 0, total = 0;
};
VarlenLayout varlen_layout(const ccq_shape* s, ccq_backbone bb, bool bwd) {
  VarlenLayout L;
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off += align_up(n);
    return o;
  };
  const size_t ntok = (size_t)s->B * s->T * s->H, e = esize(s->io_dtype), eg = esize(s->gate_dtype);
  const size_t gate = bb == CCQ_GLA ? ntok * s->dk * eg : ntok * 4;
  L.q = take(ntok * s->dk * e);
  L.k = take(ntok * s->dk * e);
  L.v = take(ntok * s->dv * e);
  L.gate = take(gate);
  if (bb == CCQ_GDN) L.beta = take(ntok * 4);
  L.lam = take(ntok * 4);
  L.o = take(ntok * s->dv * e);
  if (bwd) {
    L.dO = take(ntok * s->dv * e);
    L.dq = take(ntok * s->dk * e);
    L.dk = take(ntok * s->dk * e);
    L.dv = take(ntok * s->dv * e);
    L.dgate = take(gate);
    if (bb == CCQ_GDN) L.dbeta = take(ntok * 4);
    L.dlam = take(ntok * 4);
  }
  L.inner = off;
  const size_t inner = bwd ? (bb == CCQ_GLA ? bwd_layout(s).total : gdn_bwd_layout(s).total)
                           : fwd_layout(s, bb).total;
  L.total = off + inner;
  return L;
}

// Row bytes of the packed tensors: q/k, v, the gate (GLA [.., dk] in the gate
// dtype, Gated DeltaNet log alpha [..] fp32) and the per-head scalars.
struct VarlenRows {
  size_t qk, v, gate, scalar;
};
VarlenRows varlen_rows(const ccq_shape* s, ccq_backbone bb) {
  const size_t e = esize(s->io_dtype);
  return {(size_t)s->H * s->dk * e, (size_t)s->H * s->dv * e,
          bb == CCQ_GLA ? (size_t)s->H * s->dk * esize(s->gate_dtype) : (size_t)s->H * 4, (size_t)s->H * 4};
}

ccq_status check_varlen(const ccq_shape* s, ccq_backbone bb, const int32_t* cu) {
  ccq_status rc = check_shape(s, bb);
  if (rc != CCQ_OK) return rc;
  if (s->B > 65535) return CCQ_ERR_UNSUPPORTED;  // one grid row per sequence
  if (s->B > 0 && (!cu || (reinterpret_cast<uintptr_t>(cu) & 3u))) return CCQ_ERR_INVALID_ARG;
  return CCQ_OK;
}

ccq_status varlen_forward(ccq_backbone bb, const ccq_shape* s, const int32_t* cu, const void* q,
                          const void* k, const void* v, const void* g_or_la, const float* beta,
                          const float* lam, const float* S0, const float* C0, const float* mu0, void* o,
                          float* ST, float* CT, float* muT, void* workspace, size_t ws_bytes,
                          void* stream) {
  ccq_status rc = check_varlen(s, bb, cu);
  if (rc != CCQ_OK) return rc;
  const void* ptrs[] = {S0, C0, mu0, ST, CT, muT, workspace};
  for (const void* p : ptrs)
    if (p && !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (s->B == 0 || s->H == 0) return CCQ_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s->T == 0) return copy_initial_states(s, S0, C0, mu0, ST, CT, muT, st);
  const void* req[] = {q, k, v, g_or_la, lam, o};
  for (const void* p : req)
    if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (bb == CCQ_GDN && (!beta || !aligned(beta))) return CCQ_ERR_INVALID_ARG;
  if (!workspace || ws_bytes < fwd_layout(s, bb).total) return CCQ_ERR_WORKSPACE;
  // the kernels read the packed rows through the offsets themselves
  return run_forward(bb, s, q, k, v, g_or_la, beta, lam, S0, C0, mu0, o, ST, CT, muT, nullptr,
                     workspace, ws_bytes, stream, cu);
}

// Forward from raw q, k: the row scales 1 / |q|, 1 / |k| and the gate, then
// the forward workspace.
struct RawLayout {
  size_t rq = 0, rk = 0, lam = 0, inner = 0;
};
RawLayout raw_layout(const ccq_shape* s) {
  RawLayout L;
  const size_t n = (size_t)s->B * s->T * s->H * sizeof(float);
  L.rq = 0;
  L.rk = align_up(n);
  L.lam = 2 * align_up(n);
  L.inner = 3 * align_up(n);
  return L;
}

// Scratch of the allocation-free forward (ccq_gdn_fwd_noalloc): a device array
// of kScratchBytes, one copy on every device the library runs on, held until the
// process ends.  In host code `scratch` names a host-side stand-in, not device
// memory: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// handed to kernels.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch (looked up on its first use).
hipError_t scratch_on_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

size_t ccq_varlen_workspace_size(const ccq_shape* s, ccq_backbone bb, int with_bwd) {
  if (check_shape(s, bb) != CCQ_OK) return 0;
  if (with_bwd && !ccq::bwd_supported(s->dk, s->dv, s->io_dtype == CCQ_BF16, bb == CCQ_GDN)) return 0;
  // the forward reads packed rows directly; the training step runs on padded copies
  return with_bwd ? varlen_layout(s, bb, true).total : fwd_layout(s, bb).total;
}

ccq_status ccq_gla_fwd_varlen(const ccq_shape* s, const int32_t* cu_seqlens, const void* q, const void* k,
                              const void* v, const void* g, const float* lam, const float* S0,
                              const float* C0, const float* mu0, void* o, float* ST, float* CT, float* muT,
                              void* workspace, size_t ws_bytes, void* stream) {
  return varlen_forward(CCQ_GLA, s, cu_seqlens, q, k, v, g, nullptr, lam, S0, C0, mu0, o, ST, CT, muT,
                        workspace, ws_bytes, stream);
}

ccq_status ccq_gdn_fwd_varlen(const ccq_shape* s, const int32_t* cu_seqlens, const void* q, const void* k,
                              const void* v, const float* logalpha, const float* beta, const float* lam,
                              const float* S0, const float* C0, const float* mu0, void* o, float* ST,
                              float* CT, float* muT, void* workspace, size_t ws_bytes, void* stream) {
  return varlen_forward(CCQ_GDN, s, cu_seqlens, q, k, v, logalpha, beta, lam, S0, C0, mu0, o, ST, CT, muT,
                        workspace, ws_bytes, stream);
}

size_t ccq_workspace_size(const ccq_shape* s, ccq_backbone bb, int with_bwd) {
  if (check_shape(s, bb) != CCQ_OK) return 0;
  if (with_bwd) {
    if (!ccq::bwd_supported(s->dk, s->dv, s->io_dtype == CCQ_BF16, bb == CCQ_GDN)) return 0;
    return bb == CCQ_GLA ? bwd_layout(s).total : gdn_bwd_layout(s).total;
  }
  return fwd_layout(s, bb).total;
}

ccq_status ccq_gla_fwd(const ccq_shape* s, const void* q, const void* k, const void* v,
                       const void* g, const float* lam, const float* S0, const float* C0,
                       const float* mu0, void* o, float* ST, float* CT, float* muT,
                       float* q_clean_dbg, void* workspace, size_t ws_bytes, void* stream) {
  return run_forward(CCQ_GLA, s, q, k, v, g, nullptr, lam, S0, C0, mu0, o, ST, CT, muT,
                     q_clean_dbg, workspace, ws_bytes, stream);
}

ccq_status ccq_gdn_fwd(const ccq_shape* s, const void* q, const void* k, const void* v,
                       const float* logalpha, const float* beta, const float* lam,
                       const float* S0, const float* C0, const float* mu0, void* o, float* ST,
                       float* CT, float* muT, float* q_clean_dbg, void* workspace,
                       size_t ws_bytes, void* stream) {
  return run_forward(CCQ_GDN, s, q, k, v, logalpha, beta, lam, S0, C0, mu0, o, ST, CT, muT,
                     q_clean_dbg, workspace, ws_bytes, stream);
}

size_t ccq_fwd_raw_workspace_size(const ccq_shape* s, ccq_backbone bb) {
  if (check_shape(s, bb) != CCQ_OK || !ccq::prep_supported(s->H, s->dk)) return 0;
  return raw_layout(s).inner + fwd_layout(s, bb).total;
}

ccq_status ccq_fwd_raw(const ccq_shape* s, ccq_backbone bb, const void* q_raw, const void* k_raw,
                       const float* w_lam, const float* b_lam, const void* v,
                       const void* g_or_logalpha, const float* beta, const float* S0,
                       const float* C0, const float* mu0, void* o, float* ST, float* CT, float* muT,
                       float* lam_out, void* workspace, size_t ws_bytes, void* stream) {
  ccq_status rc = check_shape(s, bb);
  if (rc != CCQ_OK) return rc;
  const size_t ntok = (size_t)s->B * s->T * s->H;
  const void* opt[] = {S0, C0, mu0, ST, CT, muT, lam_out, workspace};
  for (const void* p : opt)
    if (p && !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (ntok > 0) {
    const void* req[] = {q_raw, k_raw, w_lam, b_lam, v, g_or_logalpha, o};
    for (const void* p : req)
      if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
    if (bb == CCQ_GDN && (!beta || !aligned(beta))) return CCQ_ERR_INVALID_ARG;
    if (!ccq::prep_supported(s->H, s->dk)) return CCQ_ERR_UNSUPPORTED;
    if ((long long)s->B * s->T / 16 >= (1LL << 31)) return CCQ_ERR_UNSUPPORTED;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s->B == 0 || s->H == 0) return CCQ_OK;
  if (s->T == 0) return copy_initial_states(s, S0, C0, mu0, ST, CT, muT, st);
  const RawLayout R = raw_layout(s);
  if (!workspace || ws_bytes < R.inner + fwd_layout(s, bb).total) return CCQ_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  float* rq = reinterpret_cast<float*>(ws + R.rq);
  float* rk = reinterpret_cast<float*>(ws + R.rk);
  float* lam = lam_out ? lam_out : reinterpret_cast<float*>(ws + R.lam);
  TraceScope scope;
  // the gate and the row scales (no normalised rows are written) ...
  ccq::PrepArgs pa{q_raw, k_raw, w_lam, b_lam, nullptr, nullptr, lam, s->B, s->T, s->H, s->dk};
  pa.rq = rq;
  pa.rk = rk;
  if (traced(st, [&] { return ccq::launch_prep(pa, s->io_dtype == CCQ_BF16, st); }) != hipSuccess)
    return CCQ_ERR_HIP;
  // ... then the forward, every kernel scaling the raw rows as it stages them
  return run_forward(bb, s, q_raw, k_raw, v, g_or_logalpha, beta, lam, S0, C0, mu0, o, ST, CT, muT,
                     nullptr, ws + R.inner, ws_bytes - R.inner, stream, nullptr, rq, rk);
}

ccq_status ccq_gdn_fwd_noalloc(const ccq_shape* s, const void* q, const void* k, const void* v,
                               const float* logalpha, const float* beta, const float* lam,
                               const float* S0, const float* C0, const float* mu0, void* o,
                               float* ST, float* CT, float* muT, float* q_clean_dbg,
                               void* stream) {
  ccq_status rc = check_forward_args(CCQ_GDN, s, q, k, v, logalpha, beta, lam, S0, C0, mu0, o,
                                     ST, CT, muT, q_clean_dbg, nullptr);
  if (rc != CCQ_OK) return rc;
  // every buffer the kernels read is written first in the same call, so the
  // previous call's contents need no clearing
  if (fwd_layout(s, CCQ_GDN).total > kScratchBytes) return CCQ_ERR_WORKSPACE;
  if (s->B == 0 || s->H == 0 || s->T == 0)  // no scratch needed
    return run_forward(CCQ_GDN, s, q, k, v, logalpha, beta, lam, S0, C0, mu0, o, ST, CT, muT,
                       q_clean_dbg, nullptr, 0, stream);
  void* ws = nullptr;
  if (scratch_on_current_device(&ws) != hipSuccess) return CCQ_ERR_HIP;
  return run_forward(CCQ_GDN, s, q, k, v, logalpha, beta, lam, S0, C0, mu0, o, ST, CT, muT,
                     q_clean_dbg, ws, kScratchBytes, stream);
}

ccq_status ccq_fwd_bwd(const ccq_shape* s, ccq_backbone bb, const void* q, const void* k,
                       const void* v, const void* g_or_logalpha, const float* beta,
                       const float* lam, const void* dO, void* o, void* dq, void* dk, void* dv,
                       void* dg_or_dlogalpha, float* dbeta, float* dlam, void* workspace,
                       size_t ws_bytes, void* stream) {
  ccq_status rc = check_shape(s, bb);
  if (rc != CCQ_OK) return rc;
  if (s->t0 != 0) return CCQ_ERR_INVALID_ARG;     // a training step starts from zero states
  if (s->decay_aligned) return CCQ_ERR_UNSUPPORTED;  // the decay-aligned statistics: forward only
  const bool bf = s->io_dtype == CCQ_BF16;
  const bool gbf = s->gate_dtype == CCQ_BF16;
  if (!ccq::bwd_supported(s->dk, s->dv, bf, bb == CCQ_GDN)) return CCQ_ERR_UNSUPPORTED;
  const size_t ntok = (size_t)s->B * s->T * s->H;
  if (workspace && !aligned(workspace)) return CCQ_ERR_INVALID_ARG;
  if (ntok > 0) {
    const void* req[] = {q, k, v, g_or_logalpha, lam, dO, o, dq, dk, dv, dg_or_dlogalpha, dlam};
    for (const void* p : req)
      if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
    if (bb == CCQ_GDN && (!beta || !aligned(beta) || !dbeta || !aligned(dbeta)))
      return CCQ_ERR_INVALID_ARG;
  }
  if (ntok == 0) return CCQ_OK;
  if (bb == CCQ_GDN)
    return gdn_fwd_bwd(s, q, k, v, static_cast<const float*>(g_or_logalpha), beta, lam, dO, o, dq,
                       dk, dv, static_cast<float*>(dg_or_dlogalpha), dbeta, dlam, workspace,
                       ws_bytes, stream);
  const BwdLayout L = bwd_layout(s);
  if (!workspace || ws_bytes < L.total) return CCQ_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* corr = reinterpret_cast<float*>(ws + L.corr);
  float* mdq = reinterpret_cast<float*>(ws + L.mdq);
  float* mdu = reinterpret_cast<float*>(ws + L.mdu);
  float* dqc = reinterpret_cast<float*>(ws + L.dqc);
  float* dkg = reinterpret_cast<float*>(ws + L.dkg);
  float* db = reinterpret_cast<float*>(ws + L.db);
  float* dgn = reinterpret_cast<float*>(ws + L.dgn);
  trace_begin_call();

  // forward: cleaned queries (with Sigma q and m.q kept), then GLA keeping S_r
  ccq::CleanArgs c1 = clean_args(s, ws, L.clean);
  c1.q = q;
  c1.k = k;
  c1.lam = lam;
  c1.qclean = ws + L.qclean;
  c1.corr = corr;
  c1.mdot = mdq;
  if (run_clean_stats(c1, bf, st) != hipSuccess) return CCQ_ERR_HIP;
  if (traced(st, [&] { return ccq::launch_clean_out(c1, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GlaStateArgs sa{k, v, g_or_logalpha, nullptr, nullptr, ws + L.states, s->B, s->T, s->H,
                       s->dk, s->dv};
  if (traced(st, [&] { return ccq::launch_gla_state(sa, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GlaOutArgs oa{ws + L.qclean, k, v, g_or_logalpha, ws + L.states, o, s->B, s->T, s->H, s->dk,
                     s->dv, s->scale};
  // every S_r is stored (the backward reads them); the output kernel still
  // reads only each group's first and carries S through the group
  oa.group = ccq::gla_out_group(s->B, s->H, s->T, s->dk, s->dv, bf);
  if (traced(st, [&] { return ccq::launch_gla_out(oa, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  // backward: dS scan, chunk gradients, decay gradient, dq, dk
  ccq::DstateArgs da{ws + L.qclean, g_or_logalpha, dO, ws + L.dstates, s->B, s->T, s->H, s->dk,
                     s->dv, s->scale};
  if (traced(st, [&] { return ccq::launch_gla_dstate(da, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::GlaBwdArgs ba{ws + L.qclean, k, v, g_or_logalpha, dO, ws + L.states, ws + L.dstates, corr,
                     dqc, ws + L.dqc_io, dkg, dv, db, dgn, dlam, s->B, s->T, s->H, s->dk, s->dv,
                     s->scale};
  if (traced(st, [&] { return ccq::launch_gla_bwd_chunk(ba, bf, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::DgArgs ga2{db, dgn, dg_or_dlogalpha, s->B, s->T, s->H, s->dk};
  if (traced(st, [&] { return ccq::launch_gla_dg(ga2, gbf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::CleanArgs c2 = clean_args(s, ws, L.clean);  // same keys: statistics reused
  c2.q = ws + L.dqc_io;
  c2.k = k;
  c2.lam = lam;
  c2.qclean = dq;
  c2.base = dqc;
  c2.mdot = mdu;
  if (traced(st, [&] { return ccq::launch_clean_out(c2, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  ccq::CcqDkArgs ka{q, k, ws + L.dqc_io, lam, mdq, mdu, dkg, dk, s->B, s->T, s->H, s->dk,
                    s->centered};
  set_dk_ws(ka, s, ws, L.dkws);
  if (traced(st, [&] { return ccq::launch_ccq_dk(ka, bf, st); }) != hipSuccess) return CCQ_ERR_HIP;
  return CCQ_OK;
}

ccq_status ccq_fwd_bwd_varlen(const ccq_shape* s, ccq_backbone bb, const int32_t* cu_seqlens, const void* q,
                              const void* k, const void* v, const void* g_or_logalpha, const float* beta,
                              const float* lam, const void* dO, void* o, void* dq, void* dk, void* dv,
                              void* dg_or_dlogalpha, float* dbeta, float* dlam, void* workspace,
                              size_t ws_bytes, void* stream) {
  ccq_status rc = check_varlen(s, bb, cu_seqlens);
  if (rc != CCQ_OK) return rc;
  if (s->t0 != 0) return CCQ_ERR_INVALID_ARG;
  if (s->decay_aligned) return CCQ_ERR_UNSUPPORTED;  // the decay-aligned statistics: forward only
  if (!ccq::bwd_supported(s->dk, s->dv, s->io_dtype == CCQ_BF16, bb == CCQ_GDN)) return CCQ_ERR_UNSUPPORTED;
  if (workspace && !aligned(workspace)) return CCQ_ERR_INVALID_ARG;
  if ((size_t)s->B * s->T * s->H == 0) return CCQ_OK;
  const void* req[] = {q, k, v, g_or_logalpha, lam, dO, o, dq, dk, dv, dg_or_dlogalpha, dlam};
  for (const void* p : req)
    if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (bb == CCQ_GDN && (!beta || !aligned(beta) || !dbeta || !aligned(dbeta))) return CCQ_ERR_INVALID_ARG;
  const VarlenLayout L = varlen_layout(s, bb, true);
  if (!workspace || ws_bytes < L.total) return CCQ_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  const VarlenRows R = varlen_rows(s, bb);
  const int32_t* cu = cu_seqlens;
  TraceScope scope;
  auto copy = [&](void* dst, const void* src, size_t rb, bool to_padded) {
    return traced(st, [&] { return ccq::launch_varlen_copy(dst, src, cu, s->B, s->T, rb, to_padded, st); }) ==
           hipSuccess;
  };
  if (!copy(ws + L.q, q, R.qk, true) || !copy(ws + L.k, k, R.qk, true) || !copy(ws + L.v, v, R.v, true) ||
      !copy(ws + L.gate, g_or_logalpha, R.gate, true) || (bb == CCQ_GDN && !copy(ws + L.beta, beta, R.scalar, true)) ||
      !copy(ws + L.lam, lam, R.scalar, true) || !copy(ws + L.dO, dO, R.v, true))
    return CCQ_ERR_HIP;
  rc = ccq_fwd_bwd(s, bb, ws + L.q, ws + L.k, ws + L.v, ws + L.gate,
                   bb == CCQ_GDN ? reinterpret_cast<const float*>(ws + L.beta) : nullptr,
                   reinterpret_cast<const float*>(ws + L.lam), ws + L.dO, ws + L.o, ws + L.dq, ws + L.dk,
                   ws + L.dv, ws + L.dgate, bb == CCQ_GDN ? reinterpret_cast<float*>(ws + L.dbeta) : nullptr,
                   reinterpret_cast<float*>(ws + L.dlam), ws + L.inner, ws_bytes - L.inner, stream);
  if (rc != CCQ_OK) return rc;
  if (!copy(o, ws + L.o, R.v, false) || !copy(dq, ws + L.dq, R.qk, false) || !copy(dk, ws + L.dk, R.qk, false) ||
      !copy(dv, ws + L.dv, R.v, false) || !copy(dg_or_dlogalpha, ws + L.dgate, R.gate, false) ||
      (bb == CCQ_GDN && !copy(dbeta, ws + L.dbeta, R.scalar, false)) || !copy(dlam, ws + L.dlam, R.scalar, false))
    return CCQ_ERR_HIP;
  return CCQ_OK;
}

// Decode workspace: Cbar_t q [B,H,dk] fp32 when the step is split into two
// launches (a few large heads), else none.
size_t ccq_decode_workspace_size(const ccq_shape* s) {
  if (!s || s->B < 0 || s->H < 0 || !ccq::decode_supported(s->dk, s->dv)) return 0;
  const long long bh = (long long)s->B * s->H;
  if (!ccq::decode_split(bh, s->dk, s->dv)) return 0;
  return align_up((size_t)bh * s->dk * sizeof(float));
}

ccq_status ccq_decode(const ccq_shape* s, ccq_backbone bb, const void* q, const void* k,
                      const void* v, const void* g_or_logalpha, const float* beta,
                      const float* lam, float* S, float* C, float* mu, void* o, void* workspace,
                      size_t ws_bytes, void* stream) {
  if (!s) return CCQ_ERR_INVALID_ARG;
  if (s->B < 0 || s->H < 0 || s->t0 < 0 || s->T != 1) return CCQ_ERR_INVALID_ARG;
  if (!dtype_ok(s->io_dtype) || !dtype_ok(s->gate_dtype)) return CCQ_ERR_INVALID_ARG;
  if (s->centered != 0 && s->centered != 1) return CCQ_ERR_INVALID_ARG;
  if (s->decay_aligned != 0 && s->decay_aligned != 1) return CCQ_ERR_INVALID_ARG;
  if (bb != CCQ_GLA && bb != CCQ_GDN) return CCQ_ERR_INVALID_ARG;
  if (s->decay_aligned) return CCQ_ERR_UNSUPPORTED;  // the cache holds no decayed count
  if (!ccq::decode_supported(s->dk, s->dv)) return CCQ_ERR_UNSUPPORTED;
  if ((long long)s->B * s->H > 0x7fffffffLL) return CCQ_ERR_UNSUPPORTED;  // one workgroup per head
  if (s->B == 0 || s->H == 0) return CCQ_OK;
  const void* req[] = {q, k, v, g_or_logalpha, lam, S, C, mu, o};
  for (const void* p : req)
    if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if (bb == CCQ_GDN && (!beta || !aligned(beta))) return CCQ_ERR_INVALID_ARG;
  const size_t need = ccq_decode_workspace_size(s);
  if (need && (!workspace || !aligned(workspace) || ws_bytes < need)) return CCQ_ERR_WORKSPACE;
  ccq::DecodeArgs a{q, k, v, g_or_logalpha, beta, lam, S, C, mu,
                    need ? static_cast<float*>(workspace) : nullptr,
                    o, s->B, s->H, s->dk, s->dv, s->centered, s->scale, s->t0};
  hipStream_t st = static_cast<hipStream_t>(stream);
  trace_begin_call();
  if (traced(st, [&] {
        return ccq::launch_decode(a, bb == CCQ_GDN, s->io_dtype == CCQ_BF16,
                                  s->gate_dtype == CCQ_BF16, st);
      }) != hipSuccess)
    return CCQ_ERR_HIP;
  return CCQ_OK;
}

ccq_status ccq_prep(const ccq_shape* s, const void* q_raw, const void* k_raw, const float* w_lam,
                    const float* b_lam, void* q, void* k, float* lam, void* stream) {
  if (!s) return CCQ_ERR_INVALID_ARG;
  if (s->B < 0 || s->T < 0 || s->H < 0) return CCQ_ERR_INVALID_ARG;
  if (!dtype_ok(s->io_dtype)) return CCQ_ERR_INVALID_ARG;
  if ((long long)s->B * s->T * s->H == 0) return CCQ_OK;
  if (!ccq::prep_supported(s->H, s->dk)) return CCQ_ERR_UNSUPPORTED;
  const void* req[] = {q_raw, k_raw, w_lam, b_lam, q, k, lam};
  for (const void* p : req)
    if (!p || !aligned(p)) return CCQ_ERR_INVALID_ARG;
  if ((long long)s->B * s->T / 16 >= (1LL << 31)) return CCQ_ERR_UNSUPPORTED;
  ccq::PrepArgs a{q_raw, k_raw, w_lam, b_lam, q, k, lam, s->B, s->T, s->H, s->dk};
  hipStream_t st = static_cast<hipStream_t>(stream);
  trace_begin_call();
  if (traced(st, [&] { return ccq::launch_prep(a, s->io_dtype == CCQ_BF16, st); }) != hipSuccess)
    return CCQ_ERR_HIP;
  return CCQ_OK;
}

ccq_status ccq_trace_events(void* const* events, int n_events) {
  if (events == nullptr || n_events <= 0) {
    g_trace = Trace{};
    return CCQ_OK;
  }
  for (int i = 0; i < n_events; ++i)
    if (!events[i]) return CCQ_ERR_INVALID_ARG;
  g_trace.ev = reinterpret_cast<hipEvent_t*>(const_cast<void**>(events));
  g_trace.n = n_events;
  g_trace.next = 0;
  return CCQ_OK;
}

const char* ccq_status_string(ccq_status st) {
  switch (st) {
    case CCQ_OK: return "ok";
    case CCQ_ERR_INVALID_ARG: return "invalid argument";
    case CCQ_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case CCQ_ERR_WORKSPACE: return "workspace missing or too small";
    case CCQ_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

const char* ccq_version(void) { return "ccq-mi355x 0.1.0 gfx950"; }

}  // extern "C"
