/*
 * ccq.h -- C ABI of the MI355X (gfx950) Curvature-Conditioned Query library.
 *
 * Curvature-Conditioned Query (CCQ, arXiv 2606.01294) cleans every query of
 * a linear-attention layer before it reads the fast-weight state:
 *
 *     Sigma_t   = Cbar_t - mu_t mu_t^T,  Cbar_t = (1/t) sum_{j<=t} k_j k_j^T,
 *                                        mu_t   = (1/t) sum_{j<=t} k_j
 *                                        (Sec. 3.2, second-order expansion)
 *     q_clean_t = q_t - lambda_t Sigma_t q_t                     (Eq. clean)
 *     o_t       = scale * S_t q_clean_t                          (Eq. read)
 *
 * where S_t is the backbone state, written before it is read.  The library
 * computes this with the chunkwise form of Alg. 1 (App. B: the second-moment
 * and mean terms split into a carried inter-chunk state and an intra-chunk
 * block) for two backbones:
 *
 *   GLA             S_t = S_{t-1} diag(exp g_t) + v_t k_t^T,   g_t in R^{dk}
 *   Gated DeltaNet  S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Every tensor argument is a DEVICE pointer owned by the caller, dense and
 *    row-major.  Token tensors are [B, T, H, d]; states are [B, H, ...].
 *    Pointers must be 16-byte aligned.
 *  * The library allocates and frees nothing.  Scratch comes from the caller's
 *    `workspace` of at least ccq_workspace_size() bytes (16-byte aligned).
 *  * Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream): every kernel of a call is launched on that stream, in order.
 *    The library creates no streams or events.  Arguments are validated
 *    before anything is launched; on an error nothing is launched and nothing
 *    is written.  A failed launch returns CCQ_ERR_HIP.  Nothing aborts,
 *    nothing throws, and nothing is kept between calls except the per-thread
 *    setting of the timing hook ccq_trace_events (off unless a caller sets
 *    it): concurrent calls on different workspaces are safe.
 *  * q and k are used as given (the caller applies any l2-normalisation, as
 *    Alg. 1 does before the cleaning lines).  NaN/Inf inputs propagate.
 *  * Statistics (Cbar, mu) and the backbone state are fp32 whatever io_dtype
 *    is; products run on the MFMA units with fp32 accumulation.
 */
#ifndef CCQ_H_
#define CCQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CCQ_OK = 0,
  CCQ_ERR_INVALID_ARG = 1, /* NULL where a tensor is required, negative sizes, misalignment */
  CCQ_ERR_UNSUPPORTED = 2, /* a head size, chunk or dtype the library has no kernel for */
  CCQ_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than ccq_workspace_size() */
  CCQ_ERR_HIP = 4          /* the HIP runtime reported an error at launch */
} ccq_status;

typedef enum { CCQ_F32 = 0, CCQ_BF16 = 1 } ccq_dtype;
typedef enum { CCQ_GLA = 0, CCQ_GDN = 1 } ccq_backbone;

typedef struct {
  int32_t B, T, H;      /* batch, tokens, heads (T may be any value >= 0) */
  int32_t dk, dv;       /* key / value head size: dv in {64,128,256,512}; dk in {64,128}
                         * (GLA, or fp32 io), {64,128,256} (bf16 Gated DeltaNet) */
  int32_t chunk;        /* chunk length C of Alg. 1; must be 64 */
  ccq_dtype io_dtype;   /* dtype of q, k, v, o (and of dq, dk, dv, dO in the backward) */
  ccq_dtype gate_dtype; /* dtype of the GLA gate g (and of dg); ignored for GDN */
  float scale;          /* o = scale * S q_clean; the paper's read uses 1.0 */
  int32_t centered;     /* 1: Sigma = Cbar - mu mu^T (the paper); 0: Sigma = Cbar (App. E ablation) */
  int32_t decay_aligned;/* 0: the paper's undecayed statistics.  1 (Gated DeltaNet forward only):
                         * the decay-aligned covariance Sigma^gamma that App. J names as future
                         * work for forgetting backbones, read as key j entering token t's
                         * statistics with the backbone's own decay prod_{s=j+1..t} alpha_s and
                         * t replaced by the decayed count W_t = alpha_t W_{t-1} + 1 (Alg. 2's
                         * running means with W_t for t); alpha = 1 gives Sigma_t.  Needs t0 = 0
                         * and no C0 / mu0 (the cache holds no W); CT, muT are then the
                         * weighted means.  Else CCQ_ERR_UNSUPPORTED (GLA, whose decay is per
                         * channel; ccq_fwd_bwd; ccq_decode). */
  int64_t t0;           /* tokens already absorbed into C0/mu0; positions are t0+1 .. t0+T */
} ccq_shape;

/* Bytes of device workspace the call needs (0 when none).  with_bwd selects
 * the training entry point ccq_fwd_bwd.  Returns 0 for an invalid shape. */
size_t ccq_workspace_size(const ccq_shape* s, ccq_backbone bb, int with_bwd);

/*
 * CCQ-GLA chunkwise forward (Alg. 1 with the GLA chunk form as BackboneUpdate).
 *   q, k     [B,T,H,dk] io_dtype      queries / keys
 *   v        [B,T,H,dv] io_dtype      values
 *   g        [B,T,H,dk] gate_dtype    per-key-channel log forget gate (<= 0)
 *   lam      [B,T,H]    fp32          contraction gate lambda_t (Eq. clean)
 *   S0       [B,H,dv,dk] fp32 or NULL initial backbone state (NULL = 0)
 *   C0       [B,H,dk,dk] fp32 or NULL initial Cbar (NULL = 0), weight t0
 *   mu0      [B,H,dk]    fp32 or NULL initial mu (NULL = 0), weight t0
 *   o        [B,T,H,dv] io_dtype      output (written)
 *   ST, CT, muT  final (S_T, Cbar_T, mu_T), the inference cache of App. C,
 *                same layouts as S0, C0, mu0; each may be NULL (not wanted)
 *   q_clean_dbg [B,T,H,dk] fp32 or NULL: the cleaned queries, for checking
 */
ccq_status ccq_gla_fwd(const ccq_shape* s, const void* q, const void* k, const void* v,
                       const void* g, const float* lam, const float* S0, const float* C0,
                       const float* mu0, void* o, float* ST, float* CT, float* muT,
                       float* q_clean_dbg, void* workspace, size_t ws_bytes, void* stream);

/*
 * CCQ-Gated-DeltaNet chunkwise forward (Alg. 1 with the delta-rule chunk form
 * computed through the WY/UT transform as BackboneUpdate).
 *   logalpha [B,T,H] fp32   log of the per-head scalar decay alpha_t (<= 0)
 *   beta     [B,T,H] fp32   write strength beta_t in [0,1]
 * All other arguments as in ccq_gla_fwd.
 */
ccq_status ccq_gdn_fwd(const ccq_shape* s, const void* q, const void* k, const void* v,
                       const float* logalpha, const float* beta, const float* lam,
                       const float* S0, const float* C0, const float* mu0, void* o, float* ST,
                       float* CT, float* muT, float* q_clean_dbg, void* workspace,
                       size_t ws_bytes, void* stream);

/*
 * Allocation-free form of ccq_gdn_fwd, for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments and results as
 * ccq_gdn_fwd without the workspace: the kernels use a scratch array of
 * CCQ_NOALLOC_SCRATCH_BYTES that the library holds in device memory, one copy
 * per device, from the first call on that device until the process ends.  The
 * call allocates nothing (no hipMalloc, hipFree or allocating library call).
 * Shapes whose ccq_workspace_size(s, CCQ_GDN, 0) exceeds
 * CCQ_NOALLOC_SCRATCH_BYTES return CCQ_ERR_WORKSPACE before anything is
 * launched (at dk = dv = 256 that is about 10,000 token-heads, B*T*H, per call).
 * All calls on one device share its scratch: calls that may overlap on one
 * device (two streams, two host threads) race and must be ordered by the
 * caller; calls ordered on one stream are safe.  The scratch keeps the last
 * call's contents, and no call reads what an earlier call left there.
 */
#define CCQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ccq_status ccq_gdn_fwd_noalloc(const ccq_shape* s, const void* q, const void* k, const void* v,
                               const float* logalpha, const float* beta, const float* lam,
                               const float* S0, const float* C0, const float* mu0, void* o,
                               float* ST, float* CT, float* muT, float* q_clean_dbg,
                               void* stream);

/*
 * Training step: forward and the gradients of L = sum_t <dO_t, o_t> with
 * respect to q, k, v, the gates and lambda (fresh sequence: zero initial
 * states, t0 must be 0).
 *   bb = CCQ_GLA: g_or_logalpha is g [B,T,H,dk] gate_dtype; beta and dbeta NULL;
 *                 dg_or_dlogalpha is dg [B,T,H,dk] gate_dtype.
 *   bb = CCQ_GDN: g_or_logalpha is log alpha [B,T,H] fp32 and beta [B,T,H]
 *                 fp32 is required; dg_or_dlogalpha is d(log alpha) [B,T,H]
 *                 fp32 and dbeta [B,T,H] fp32 is required.  The backbone
 *                 gradients follow the reverse of the chunk form through the
 *                 WY/UT transform (Alg. 1's BackboneUpdate for the delta rule).
 *   dO [B,T,H,dv] io_dtype upstream gradient; o, dq, dk, dv io_dtype;
 *   dlam [B,T,H] fp32.
 * Supported: chunk = 64, dv in {64,128,256,512}, and dk in {64,128} for bf16
 * io (also 256 for CCQ_GDN) or dk = 64 for fp32 io; other shapes return
 * CCQ_ERR_UNSUPPORTED.
 */
ccq_status ccq_fwd_bwd(const ccq_shape* s, ccq_backbone bb, const void* q, const void* k,
                       const void* v, const void* g_or_logalpha, const float* beta,
                       const float* lam, const void* dO, void* o, void* dq, void* dk, void* dv,
                       void* dg_or_dlogalpha, float* dbeta, float* dlam, void* workspace,
                       size_t ws_bytes, void* stream);

/*
 * Recurrent inference, one token per sequence (Alg. 2), on the cache triple
 * of App. C, updated in place:
 *   Cbar <- Cbar + (k k^T - Cbar)/t,  mu <- mu + (k - mu)/t,  t = s->t0 + 1;
 *   q_clean = q - lam (Cbar q - mu (mu . q))   (Cbar q alone when centered = 0);
 *   S <- BackboneUpdate(S; k, v, gates);  o = scale S q_clean.
 * s->T must be 1; s->t0 is the number of tokens already absorbed (the cache of
 * a fresh sequence is all zeros with t0 = 0).  q, k [B,H,dk] and v, o [B,H,dv]
 * in io_dtype (one token, T = 1, of the [B,T,H,d] layout); GLA gate g [B,H,dk]
 * gate_dtype; Gated DeltaNet log alpha and beta [B,H] fp32 (beta NULL for GLA);
 * lam [B,H] fp32.  S [B,H,dv,dk], C [B,H,dk,dk] and mu [B,H,dk] are fp32,
 * caller-owned, read and overwritten.  Supported: dk in {64,128,256}, dv in
 * {64,128,256,512}, both backbones and both io dtypes.
 * The workspace holds ccq_decode_workspace_size(s) bytes, B*H*dk*4 rounded
 * up when the step is split into two launches (fewer than 256 heads of large
 * caches), else 0, and workspace may then be NULL.
 */
size_t ccq_decode_workspace_size(const ccq_shape* s);
ccq_status ccq_decode(const ccq_shape* s, ccq_backbone bb, const void* q, const void* k,
                      const void* v, const void* g_or_logalpha, const float* beta,
                      const float* lam, float* S, float* C, float* mu, void* o, void* workspace,
                      size_t ws_bytes, void* stream);

/*
 * Pre-processing of one layer's raw queries and keys (Alg. 1: the per-chunk
 * l2 normalisation of Q and K, and the gate Lambda = sigma(Q W_lambda^T +
 * b_lambda) computed from the query before normalisation; Eq. clean):
 *   q[b,t,h,:] = q_raw[b,t,h,:] / max(|q_raw[b,t,h,:]|, 1e-12), k likewise;
 *   lam[b,t,h] = sigmoid(sum_j w_lam[h][j] q_raw[b,t,j] + b_lam[h]),
 * where j runs over all H*dk features of the token's query before the split
 * into heads (head-major).  q_raw, k_raw, q, k [B,T,H,dk] io_dtype; w_lam
 * [H, H*dk] fp32; b_lam [H] fp32; lam [B,T,H] fp32.  q and k may be q_raw and
 * k_raw (in place).  Uses s->B, T, H, dk and io_dtype.  Supported: dk in
 * {64,128,256}, H <= 16, H*dk <= 2048 and H*H*dk <= 16384 (W_lambda is
 * staged on chip); otherwise CCQ_ERR_UNSUPPORTED.  Allocates nothing.
 */
ccq_status ccq_prep(const ccq_shape* s, const void* q_raw, const void* k_raw, const float* w_lam,
                    const float* b_lam, void* q, void* k, float* lam, void* stream);

/*
 * Forward from the raw queries and keys: Alg. 1's per-chunk l2 normalisation
 * of Q and K and the gate Lambda = sigma(Q W_lambda^T + b_lambda) (Eq. clean)
 * folded into the forward, with the results of ccq_prep followed by
 * ccq_gla_fwd (bb = CCQ_GLA) or ccq_gdn_fwd (bb = CCQ_GDN), but without the
 * normalised q and k ever being written: a first pass reads the raw rows once
 * and writes only the per-row scales 1 / max(|x|, 1e-12) and the gate
 * (3 floats per token and head, in the workspace), and every kernel of the
 * forward scales the raw rows as it stages them.
 *   q_raw, k_raw [B,T,H,dk] io_dtype; w_lam [H, H*dk] fp32; b_lam [H] fp32 (as
 *   ccq_prep); v, the gates, S0, C0, mu0, o, ST, CT, muT as in the forward
 *   entry points (beta required for CCQ_GDN, NULL for CCQ_GLA);
 *   lam_out [B,T,H] fp32 or NULL: the gate, if the caller wants it.
 * The workspace holds ccq_fwd_raw_workspace_size(s, bb) bytes (0 for an
 * unsupported shape).  Shape limits are those of both the forward and
 * ccq_prep (H <= 16, H*dk <= 2048, H*H*dk <= 16384); q_clean export is not
 * offered here.
 */
size_t ccq_fwd_raw_workspace_size(const ccq_shape* s, ccq_backbone bb);
ccq_status ccq_fwd_raw(const ccq_shape* s, ccq_backbone bb, const void* q_raw, const void* k_raw,
                       const float* w_lam, const float* b_lam, const void* v,
                       const void* g_or_logalpha, const float* beta, const float* S0,
                       const float* C0, const float* mu0, void* o, float* ST, float* CT, float* muT,
                       float* lam_out, void* workspace, size_t ws_bytes, void* stream);

/*
 * Packed batches of sequences of different lengths: Alg. 1 (and its
 * training step) applied to every sequence on its own, each an independent
 * recurrence with its own states, exactly as if each were a call of its own.
 * Sequence b occupies rows cu_seqlens[b] .. cu_seqlens[b+1] - 1 of the packed
 * tensors: q, k, dq, dk [rows,H,dk] and v, o, dO, dv [rows,H,dv] in io_dtype,
 * the GLA gate g / dg [rows,H,dk] in gate_dtype, Gated DeltaNet log alpha,
 * beta and their gradients [rows,H] fp32, lam / dlam [rows,H] fp32.
 * cu_seqlens is a DEVICE array of B + 1 int32 (0 = cu[0] <= cu[1] <= ...);
 * s->B is the number of sequences and s->T an upper bound on their lengths
 * (a longer sequence is cut at T; the device offsets are not validated by
 * the host: the packed tensors must hold cu[B] rows).  S0, C0, mu0, ST, CT,
 * muT are per sequence, as in the padded calls; a sequence of length 0 with
 * t0 = 0 returns its initial states (or zeros).  The forward kernels read and
 * write the packed rows directly, through the offsets, and walk only each
 * sequence's own chunks.  The training step lays the sequences out as a
 * padded [B,T,...] batch in the workspace (rows past a sequence's end are
 * zero, which leaves every state unchanged and no output of the sequence's
 * own rows), runs the padded path and copies the results back.  q_clean
 * export is not offered here.  The workspace holds
 * ccq_varlen_workspace_size(s, bb, with_bwd) bytes (0: unsupported shape):
 * the padded call's for the forward, plus the padded copies for training.
 * Errors as for the padded entry points; B > 65535 is CCQ_ERR_UNSUPPORTED.
 */
size_t ccq_varlen_workspace_size(const ccq_shape* s, ccq_backbone bb, int with_bwd);
ccq_status ccq_gla_fwd_varlen(const ccq_shape* s, const int32_t* cu_seqlens, const void* q,
                              const void* k, const void* v, const void* g, const float* lam,
                              const float* S0, const float* C0, const float* mu0, void* o,
                              float* ST, float* CT, float* muT, void* workspace, size_t ws_bytes,
                              void* stream);
ccq_status ccq_gdn_fwd_varlen(const ccq_shape* s, const int32_t* cu_seqlens, const void* q,
                              const void* k, const void* v, const float* logalpha,
                              const float* beta, const float* lam, const float* S0,
                              const float* C0, const float* mu0, void* o, float* ST, float* CT,
                              float* muT, void* workspace, size_t ws_bytes, void* stream);
/* Training step on a packed batch (as ccq_fwd_bwd, t0 = 0). */
ccq_status ccq_fwd_bwd_varlen(const ccq_shape* s, ccq_backbone bb, const int32_t* cu_seqlens,
                              const void* q, const void* k, const void* v,
                              const void* g_or_logalpha, const float* beta, const float* lam,
                              const void* dO, void* o, void* dq, void* dk, void* dv,
                              void* dg_or_dlogalpha, float* dbeta, float* dlam, void* workspace,
                              size_t ws_bytes, void* stream);

/*
 * Per-kernel timing hook (instrumentation for benchmarks and profilers, not
 * part of the method).  `events` points at n_events hipEvent_t handles created
 * by the caller (hipEventCreate).  Until the next ccq_trace_events call from
 * the same host thread, every entry point called from that thread records
 * events[2i] on its stream just before its i-th kernel launch and
 * events[2i+1] just after it, for i < n_events/2; the count restarts at each
 * entry-point call.  events = NULL (or n_events = 0) switches tracing off.
 * The setting is per host thread; nothing else is kept between calls.
 */
ccq_status ccq_trace_events(void* const* events, int n_events);

/* Human-readable text of a status code (static storage). */
const char* ccq_status_string(ccq_status st);

/* Library version string, e.g. "ccq-mi355x 0.1.0 gfx950". */
const char* ccq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CCQ_H_ */
