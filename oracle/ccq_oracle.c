/*
 * ccq_oracle.c -- plain fp64 CPU oracle for Curvature-Conditioned Query (CCQ).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the HIP library; the two meet only through the seeded inputs.
 *
 * What it computes (paper: "Curvature-Conditioned Query", arXiv 2606.01294):
 *   - running key statistics  Cbar_t = (1/t) sum_{j<=t} k_j k_j^T,
 *     mu_t = (1/t) sum_{j<=t} k_j, Sigma_t = Cbar_t - mu_t mu_t^T
 *     (Sec. 3.2, second-order expansion of A_t; App. A.2);
 *   - the cleaned query q_clean = q - lambda_t Sigma_t q      (Eq. clean);
 *   - the read o_t = S_t q_clean with the backbone state S_t (Eq. read),
 *     the write happening before the read (Eq. prelim_linattn);
 *   - backbones: GLA, S_t = S_{t-1} diag(exp g_t) + v_t k_t^T, and Gated
 *     DeltaNet, S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     (the cited GLA and Gated DeltaNet papers; the paper treats the backbone
 *     as a black box, Sec. 2.2).
 *
 * Three forward forms:
 *   form 0: token-by-token recurrence on the raw sums K_t = sum k k^T and
 *           m_t = sum k, divided by t at use (App. B divides by t only once
 *           the product with the query is formed);
 *   form 1: Alg. 2 (recurrent inference), running-mean updates of Cbar, mu;
 *   chunk : Alg. 1 (chunkwise forward), with the backbone's chunk forms.
 * and two reverse passes (GLA + CCQ, Gated DeltaNet + CCQ), recomputing each
 * segment from checkpointed states.
 *
 * Readings where the paper is silent or garbled (each also recorded in the
 * design notes):
 *   * Sigma_t includes the current key k_t (Alg. 2 updates Cbar before the
 *     read; the intra-chunk sum in App. B runs over rC < j <= t).
 *   * t is the 1-based absolute position including t0 tokens absorbed into
 *     the initial statistics C0, mu0.
 *   * Alg. 1's MeanCorr term is row-wise: CumK_i (CumK_i . q_i) / t_i^2
 *     (App. B, mean term), and P^prev's row i is S^K_r q_i.
 *   * centered = 0 selects the uncentred ablation Sigma := Cbar (App. E).
 *   * o is multiplied by `scale` (1.0 reproduces the paper).
 *   * decay = 1 selects the decay-aligned covariance Sigma^gamma that App. J
 *     names as future work for forgetting backbones, read for the scalar decay
 *     of Gated DeltaNet: key j enters the statistics of token t with the
 *     backbone's own factor gamma_{j,t} = prod_{s=j+1..t} alpha_s, normalised
 *     by the decayed count W_t = sum_{j<=t} gamma_{j,t} = alpha_t W_{t-1} + 1:
 *       Cbar^gamma_t = (1/W_t) sum_j gamma_{j,t} k_j k_j^T,
 *       mu^gamma_t   = (1/W_t) sum_j gamma_{j,t} k_j,
 *       Sigma^gamma_t = Cbar^gamma_t - mu^gamma_t mu^gamma_t^T,
 *     i.e. Alg. 2's running-mean updates with t replaced by W_t.  With
 *     alpha = 1 this is Sigma_t.  Forward only, from empty statistics (t0 = 0,
 *     no C0 / mu0); CT, muT are then Cbar^gamma_T, mu^gamma_T.
 *
 * Layouts: q,k [B,T,H,dk]; v,o [B,T,H,dv]; GLA g [B,T,H,dk]; GDN logalpha,
 * beta [B,T,H]; lambda [B,T,H]; states S [B,H,dv,dk], C [B,H,dk,dk],
 * mu [B,H,dk].  All row-major fp64.  NULL initial states mean zero.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
  int32_t B, T, H, dk, dv;
  int32_t backbone; /* 0 = GLA, 1 = Gated DeltaNet */
  int32_t centered; /* 1 = Sigma = Cbar - mu mu^T, 0 = Cbar */
  int32_t decay;    /* 1 = decay-aligned statistics (Gated DeltaNet), 0 = undecayed */
  double scale;     /* read scale */
  int64_t t0;       /* tokens already absorbed into C0, mu0 */
} ccq_oracle_shape;

static size_t tok(const ccq_oracle_shape* s, int b, int t, int h) {
  return ((size_t)b * s->T + t) * s->H + h;
}

int ccq_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Load the initial statistics of one (b,h) as raw sums: K = t0 * C0,
 * m = t0 * mu0, S = S0 (zeros where the pointer is NULL). */
static void load_initial(const ccq_oracle_shape* s, int bh, const double* S0, const double* C0,
                         const double* mu0, double* S, double* K, double* m) {
  const int dk = s->dk, dv = s->dv;
  const double t0 = (double)s->t0;
  for (int i = 0; i < dv * dk; ++i) S[i] = S0 ? S0[(size_t)bh * dv * dk + i] : 0.0;
  for (int i = 0; i < dk * dk; ++i) K[i] = C0 ? t0 * C0[(size_t)bh * dk * dk + i] : 0.0;
  for (int i = 0; i < dk; ++i) m[i] = mu0 ? t0 * mu0[(size_t)bh * dk + i] : 0.0;
}

/* One backbone write S_t = Update(S_{t-1}; k_t, v_t, gates).  y is dv scratch. */
static void backbone_write(const ccq_oracle_shape* s, double* S, const double* k, const double* v,
                           const double* g, double logalpha, double beta, double* y) {
  const int dk = s->dk, dv = s->dv;
  if (s->backbone == 0) {
    /* GLA: S <- S diag(exp g) + v k^T (per key-channel forget gate). */
    for (int r = 0; r < dv; ++r)
      for (int a = 0; a < dk; ++a) S[r * dk + a] = S[r * dk + a] * exp(g[a]) + v[r] * k[a];
  } else {
    /* Gated DeltaNet: S <- alpha S (I - beta k k^T) + beta v k^T
     *                    = alpha S - alpha beta (S k) k^T + beta v k^T. */
    const double alpha = exp(logalpha);
    for (int r = 0; r < dv; ++r) {
      double acc = 0.0;
      for (int a = 0; a < dk; ++a) acc += S[r * dk + a] * k[a];
      y[r] = acc;
    }
    for (int r = 0; r < dv; ++r)
      for (int a = 0; a < dk; ++a)
        S[r * dk + a] = alpha * S[r * dk + a] - alpha * beta * y[r] * k[a] + beta * v[r] * k[a];
  }
}

/*
 * Token-by-token forward.  form 0: raw sums; form 1: Alg. 2 running means.
 * Outputs: o [B,T,H,dv]; optional ST, CT, muT (final normalised triple, the
 * inference cache of App. C) and qclean [B,T,H,dk].
 */
int ccq_oracle_fwd(const ccq_oracle_shape* s, int form, const double* q, const double* k,
                   const double* v, const double* gate, const double* beta, const double* lam,
                   const double* S0, const double* C0, const double* mu0, double* o, double* ST,
                   double* CT, double* muT, double* qclean) {
  if (!s || s->B < 0 || s->T < 0 || s->H < 0 || s->dk <= 0 || s->dv <= 0 || s->t0 < 0) return 1;
  if (s->backbone == 1 && !beta) return 1;
  if (s->decay && (s->backbone != 1 || s->t0 != 0 || C0 || mu0)) return 1;
  const int B = s->B, T = s->T, H = s->H, dk = s->dk, dv = s->dv;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    double* S = malloc(sizeof(double) * dv * dk);
    double* K = malloc(sizeof(double) * dk * dk); /* raw sum (form 0) or Cbar (form 1) */
    double* m = malloc(sizeof(double) * dk);      /* raw sum (form 0) or mu (form 1)   */
    double* c = malloc(sizeof(double) * dk);
    double* qc = malloc(sizeof(double) * dk);
    double* y = malloc(sizeof(double) * dv);
    if (!S || !K || !m || !c || !qc || !y) {
#pragma omp atomic write
      err = 2;
    } else {
      load_initial(s, bh, S0, C0, mu0, S, K, m);
      if (form == 1) { /* running means start from the given normalised stats */
        for (int i = 0; i < dk * dk; ++i) K[i] = C0 ? C0[(size_t)bh * dk * dk + i] : 0.0;
        for (int i = 0; i < dk; ++i) m[i] = mu0 ? mu0[(size_t)bh * dk + i] : 0.0;
      }
      double tau = (double)s->t0;
      for (int t = 0; t < T; ++t) {
        const size_t ti = tok(s, b, t, h);
        const double* kt = k + ti * dk;
        const double* qt = q + ti * dk;
        /* the weight of every earlier key falls by alpha_t (decay = 1) */
        const double al = s->decay ? exp(gate[ti]) : 1.0;
        tau = al * tau + 1.0;
        /* statistics include the current key (Alg. 2 updates before the read) */
        if (form == 0) {
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb) K[a * dk + bb] = al * K[a * dk + bb] + kt[a] * kt[bb];
          for (int a = 0; a < dk; ++a) m[a] = al * m[a] + kt[a];
          /* c = Sigma_t q = (K q)/t - m (m.q)/t^2 */
          double mq = 0.0;
          for (int a = 0; a < dk; ++a) mq += m[a] * qt[a];
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb) acc += K[a * dk + bb] * qt[bb];
            c[a] = acc / tau - (s->centered ? m[a] * mq / (tau * tau) : 0.0);
          }
        } else {
          /* Alg. 2: Cbar <- Cbar + (k k^T - Cbar)/t ; mu <- mu + (k - mu)/t */
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb)
              K[a * dk + bb] += (kt[a] * kt[bb] - K[a * dk + bb]) / tau;
          for (int a = 0; a < dk; ++a) m[a] += (kt[a] - m[a]) / tau;
          /* Sigma = Cbar - mu mu^T ; c = Sigma q */
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb)
              acc += (K[a * dk + bb] - (s->centered ? m[a] * m[bb] : 0.0)) * qt[bb];
            c[a] = acc;
          }
        }
        const double l = lam[ti];
        for (int a = 0; a < dk; ++a) qc[a] = qt[a] - l * c[a]; /* Eq. clean */
        if (qclean)
          for (int a = 0; a < dk; ++a) qclean[ti * dk + a] = qc[a];
        const double* g = s->backbone == 0 ? gate + ti * dk : NULL;
        const double la = s->backbone == 1 ? gate[ti] : 0.0;
        const double be = s->backbone == 1 ? beta[ti] : 0.0;
        backbone_write(s, S, kt, v + ti * dv, g, la, be, y);
        for (int r = 0; r < dv; ++r) { /* Eq. read: o = S_t q_clean */
          double acc = 0.0;
          for (int a = 0; a < dk; ++a) acc += S[r * dk + a] * qc[a];
          o[ti * dv + r] = s->scale * acc;
        }
      }
      /* final normalised triple (S_T, Cbar_T, mu_T) */
      if (ST) memcpy(ST + (size_t)bh * dv * dk, S, sizeof(double) * dv * dk);
      for (int i = 0; i < dk * dk; ++i) {
        double val;
        if (form == 1) val = K[i];
        else val = tau > 0.0 ? K[i] / tau : (C0 ? C0[(size_t)bh * dk * dk + i] : 0.0);
        if (CT) CT[(size_t)bh * dk * dk + i] = val;
      }
      for (int i = 0; i < dk; ++i) {
        double val;
        if (form == 1) val = m[i];
        else val = tau > 0.0 ? m[i] / tau : (mu0 ? mu0[(size_t)bh * dk + i] : 0.0);
        if (muT) muT[(size_t)bh * dk + i] = val;
      }
    }
    free(S); free(K); free(m); free(c); free(qc); free(y);
  }
  return err;
}

/* GLA chunk form of the backbone update (one chunk of n rows, S: dv x dk).
 * b_i = sum_{s<=i} g_s per key channel (inclusive, chunk-local):
 *   o_i   = S_0 (qc_i * e^{b_i}) + sum_{j<=i} [sum_c qc_i[c] k_j[c] e^{b_i[c]-b_j[c]}] v_j
 *   S_new = S_0 diag(e^{b_n}) + sum_j v_j (k_j * e^{b_n - b_j})^T                      */
static void gla_chunk(int n, int dk, int dv, double scale, const double* Qc, const double* Kc,
                      const double* Vc, const double* Gc, double* S, double* Oc, double* bcum) {
  for (int c = 0; c < dk; ++c) {
    double acc = 0.0;
    for (int i = 0; i < n; ++i) { acc += Gc[i * dk + c]; bcum[i * dk + c] = acc; }
  }
  for (int i = 0; i < n; ++i) {
    for (int r = 0; r < dv; ++r) {
      double acc = 0.0;
      for (int c = 0; c < dk; ++c) acc += S[r * dk + c] * Qc[i * dk + c] * exp(bcum[i * dk + c]);
      Oc[i * dv + r] = acc;
    }
    for (int j = 0; j <= i; ++j) {
      double w = 0.0;
      for (int c = 0; c < dk; ++c)
        w += Qc[i * dk + c] * Kc[j * dk + c] * exp(bcum[i * dk + c] - bcum[j * dk + c]);
      for (int r = 0; r < dv; ++r) Oc[i * dv + r] += w * Vc[j * dv + r];
    }
    for (int r = 0; r < dv; ++r) Oc[i * dv + r] *= scale;
  }
  const double* bn = bcum + (size_t)(n - 1) * dk;
  for (int r = 0; r < dv; ++r)
    for (int c = 0; c < dk; ++c) {
      double acc = S[r * dk + c] * exp(bn[c]);
      for (int j = 0; j < n; ++j) acc += Vc[j * dv + r] * Kc[j * dk + c] * exp(bn[c] - bcum[j * dk + c]);
      S[r * dk + c] = acc;
    }
}

/* Gated DeltaNet chunk form via the WY/UT transform (one chunk of n rows).
 * gamma_i = sum_{s<=i} log alpha_s;  A_ij = beta_i e^{gamma_i-gamma_j} (k_i.k_j), j<i;
 * Tm = (I + A)^{-1};  Ut = Tm diag(beta) V;  W = Tm diag(beta e^gamma) K;
 * U = Ut - W S_0^T;   o_i = e^{gamma_i} S_0 qc_i + sum_{j<=i} e^{gamma_i-gamma_j}(k_j.qc_i) u_j;
 * S_new = e^{gamma_n} S_0 + sum_j e^{gamma_n-gamma_j} u_j k_j^T.                         */
static void gdn_chunk(int n, int dk, int dv, double scale, const double* Qc, const double* Kc,
                      const double* Vc, const double* La, const double* Be, double* S, double* Oc,
                      double* work) {
  double* gam = work;             /* n */
  double* A = gam + n;            /* n x n */
  double* Tm = A + n * n;         /* n x n */
  double* Ut = Tm + n * n;        /* n x dv */
  double* W = Ut + (size_t)n * dv; /* n x dk */
  double* U = W + (size_t)n * dk; /* n x dv */
  double acc = 0.0;
  for (int i = 0; i < n; ++i) { acc += La[i]; gam[i] = acc; }
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < n; ++j) {
      double kk = 0.0;
      if (j < i)
        for (int c = 0; c < dk; ++c) kk += Kc[i * dk + c] * Kc[j * dk + c];
      A[i * n + j] = j < i ? Be[i] * exp(gam[i] - gam[j]) * kk : 0.0;
    }
  /* Tm = (I + A)^{-1} by forward substitution, column by column. */
  for (int col = 0; col < n; ++col)
    for (int i = 0; i < n; ++i) {
      double x = (i == col) ? 1.0 : 0.0;
      for (int j = 0; j < i; ++j) x -= A[i * n + j] * Tm[j * n + col];
      Tm[i * n + col] = x;
    }
  for (int i = 0; i < n; ++i) {
    for (int r = 0; r < dv; ++r) {
      double a2 = 0.0;
      for (int j = 0; j < n; ++j) a2 += Tm[i * n + j] * Be[j] * Vc[j * dv + r];
      Ut[i * dv + r] = a2;
    }
    for (int c = 0; c < dk; ++c) {
      double a2 = 0.0;
      for (int j = 0; j < n; ++j) a2 += Tm[i * n + j] * Be[j] * exp(gam[j]) * Kc[j * dk + c];
      W[i * dk + c] = a2;
    }
  }
  for (int i = 0; i < n; ++i)
    for (int r = 0; r < dv; ++r) {
      double ws = 0.0;
      for (int c = 0; c < dk; ++c) ws += W[i * dk + c] * S[r * dk + c];
      U[i * dv + r] = Ut[i * dv + r] - ws;
    }
  for (int i = 0; i < n; ++i) {
    for (int r = 0; r < dv; ++r) {
      double a2 = 0.0;
      for (int c = 0; c < dk; ++c) a2 += S[r * dk + c] * Qc[i * dk + c];
      Oc[i * dv + r] = exp(gam[i]) * a2;
    }
    for (int j = 0; j <= i; ++j) {
      double kq = 0.0;
      for (int c = 0; c < dk; ++c) kq += Kc[j * dk + c] * Qc[i * dk + c];
      const double w = exp(gam[i] - gam[j]) * kq;
      for (int r = 0; r < dv; ++r) Oc[i * dv + r] += w * U[j * dv + r];
    }
    for (int r = 0; r < dv; ++r) Oc[i * dv + r] *= scale;
  }
  for (int r = 0; r < dv; ++r)
    for (int c = 0; c < dk; ++c) {
      double a2 = exp(gam[n - 1]) * S[r * dk + c];
      for (int j = 0; j < n; ++j) a2 += exp(gam[n - 1] - gam[j]) * U[j * dv + r] * Kc[j * dk + c];
      S[r * dk + c] = a2;
    }
}

/*
 * Alg. 1 (CCQ chunkwise forward), chunk length C (the last chunk may be
 * shorter).  Per chunk r with t tokens before it:
 *   P^prev_i  = S^K_r q_i
 *   P^intra   = (Q K^T (.) Mask_incl) K
 *   CumK_i    = M_r + sum_{j<=i} k_j
 *   D_i       = 1/(t+i)
 *   MeanCorr_i= D_i^2 CumK_i (CumK_i . q_i)
 *   Qc        = Q - Lambda (.) (D (P^prev + P^intra) - MeanCorr)
 *   (O, S)    = BackboneUpdate(Qc, K, V, S)
 *   S^K_{r+1} = S^K_r + K^T K ;  M_{r+1} = M_r + sum_j k_j
 */
int ccq_oracle_chunk_fwd(const ccq_oracle_shape* s, int C, const double* q, const double* k,
                         const double* v, const double* gate, const double* beta,
                         const double* lam, const double* S0, const double* C0,
                         const double* mu0, double* o, double* ST, double* CT, double* muT,
                         double* qclean) {
  if (s && s->decay) return 1; /* the decay-aligned statistics: token forward only */
  if (!s || C <= 0 || s->B < 0 || s->T < 0 || s->H < 0 || s->dk <= 0 || s->dv <= 0) return 1;
  if (s->backbone == 1 && !beta) return 1;
  const int B = s->B, T = s->T, H = s->H, dk = s->dk, dv = s->dv;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    double* S = malloc(sizeof(double) * dv * dk);
    double* SK = malloc(sizeof(double) * dk * dk);
    double* M = malloc(sizeof(double) * dk);
    double* Qb = malloc(sizeof(double) * C * dk);
    double* Kb = malloc(sizeof(double) * C * dk);
    double* Vb = malloc(sizeof(double) * C * dv);
    double* Gb = malloc(sizeof(double) * C * dk);
    double* Lb = malloc(sizeof(double) * C);
    double* Bb = malloc(sizeof(double) * C);
    double* Qc = malloc(sizeof(double) * C * dk);
    double* Ob = malloc(sizeof(double) * C * dv);
    double* Amat = malloc(sizeof(double) * C * C);
    double* cum = malloc(sizeof(double) * C * dk);
    double* work = malloc(sizeof(double) * ((size_t)C + 2 * C * C + (size_t)C * (2 * dv + 2 * dk)));
    if (!S || !SK || !M || !Qb || !Kb || !Vb || !Gb || !Lb || !Bb || !Qc || !Ob || !Amat || !cum || !work) {
#pragma omp atomic write
      err = 2;
    } else {
      load_initial(s, bh, S0, C0, mu0, S, SK, M);
      double tpos = (double)s->t0;
      for (int r0 = 0; r0 < T; r0 += C) {
        const int n = (T - r0) < C ? (T - r0) : C;
        for (int i = 0; i < n; ++i) {
          const size_t ti = tok(s, b, r0 + i, h);
          memcpy(Qb + i * dk, q + ti * dk, sizeof(double) * dk);
          memcpy(Kb + i * dk, k + ti * dk, sizeof(double) * dk);
          memcpy(Vb + i * dv, v + ti * dv, sizeof(double) * dv);
          if (s->backbone == 0) memcpy(Gb + i * dk, gate + ti * dk, sizeof(double) * dk);
          else { Gb[i] = gate[ti]; Bb[i] = beta[ti]; }
          Lb[i] = lam[ti];
        }
        /* intra-chunk masked score block A = Q K^T (.) Mask_incl */
        for (int i = 0; i < n; ++i)
          for (int j = 0; j < n; ++j) {
            double acc = 0.0;
            if (j <= i)
              for (int a = 0; a < dk; ++a) acc += Qb[i * dk + a] * Kb[j * dk + a];
            Amat[i * C + j] = acc;
          }
        /* CumK = M_r + cumsum(K) */
        for (int a = 0; a < dk; ++a) {
          double acc = M[a];
          for (int i = 0; i < n; ++i) { acc += Kb[i * dk + a]; cum[i * dk + a] = acc; }
        }
        for (int i = 0; i < n; ++i) {
          const double D = 1.0 / (tpos + i + 1);
          double cq = 0.0;
          for (int a = 0; a < dk; ++a) cq += cum[i * dk + a] * Qb[i * dk + a];
          for (int a = 0; a < dk; ++a) {
            double pprev = 0.0, pintra = 0.0;
            for (int bb = 0; bb < dk; ++bb) pprev += SK[a * dk + bb] * Qb[i * dk + bb];
            for (int j = 0; j <= i; ++j) pintra += Amat[i * C + j] * Kb[j * dk + a];
            const double meancorr = s->centered ? D * D * cum[i * dk + a] * cq : 0.0;
            Qc[i * dk + a] = Qb[i * dk + a] - Lb[i] * (D * (pprev + pintra) - meancorr);
          }
        }
        if (qclean)
          for (int i = 0; i < n; ++i)
            memcpy(qclean + tok(s, b, r0 + i, h) * dk, Qc + i * dk, sizeof(double) * dk);
        if (s->backbone == 0) gla_chunk(n, dk, dv, s->scale, Qc, Kb, Vb, Gb, S, Ob, work);
        else gdn_chunk(n, dk, dv, s->scale, Qc, Kb, Vb, Gb, Bb, S, Ob, work);
        for (int i = 0; i < n; ++i)
          memcpy(o + tok(s, b, r0 + i, h) * dv, Ob + i * dv, sizeof(double) * dv);
        for (int a = 0; a < dk; ++a)
          for (int bb = 0; bb < dk; ++bb) {
            double acc = 0.0;
            for (int i = 0; i < n; ++i) acc += Kb[i * dk + a] * Kb[i * dk + bb];
            SK[a * dk + bb] += acc;
          }
        for (int a = 0; a < dk; ++a) {
          double acc = 0.0;
          for (int i = 0; i < n; ++i) acc += Kb[i * dk + a];
          M[a] += acc;
        }
        tpos += n;
      }
      if (ST) memcpy(ST + (size_t)bh * dv * dk, S, sizeof(double) * dv * dk);
      for (int i = 0; i < dk * dk; ++i)
        if (CT) CT[(size_t)bh * dk * dk + i] = tpos > 0 ? SK[i] / tpos : (C0 ? C0[(size_t)bh * dk * dk + i] : 0.0);
      for (int i = 0; i < dk; ++i)
        if (muT) muT[(size_t)bh * dk + i] = tpos > 0 ? M[i] / tpos : (mu0 ? mu0[(size_t)bh * dk + i] : 0.0);
    }
    free(S); free(SK); free(M); free(Qb); free(Kb); free(Vb); free(Gb); free(Lb); free(Bb);
    free(Qc); free(Ob); free(Amat); free(cum); free(work);
  }
  return err;
}

/*
 * Reverse pass of CCQ-GLA for the loss L = sum_t <dO_t, o_t> (fresh start:
 * zero initial states, t0 = 0).  Forward per token (tau = t):
 *   K_t = K_{t-1} + k_t k_t^T,  m_t = m_{t-1} + k_t
 *   c_t = K_t q_t / tau - m_t (m_t.q_t)/tau^2,   qc_t = q_t - lam_t c_t
 *   S_t = S_{t-1} diag(e^{g_t}) + v_t k_t^T,      o_t = scale S_t qc_t
 * Reverse, t = T..1, with adjoints dS (dv x dk), dK (dk x dk), dm (dk):
 *   dS  += scale dO_t qc_t^T ;       dqc = scale S_t^T dO_t
 *   dlam_t = -dqc . c_t ;            dc  = -lam_t dqc
 *   dq_t = dqc + K_t dc / tau - m_t (m_t . dc) / tau^2
 *   dK  += dc q_t^T / tau ;          dm  -= (dc (m_t.q_t) + q_t (m_t.dc)) / tau^2
 *   dv_t = dS k_t ;                  dk_t = dS^T v_t + (dK + dK^T) k_t + dm
 *   dg_t[c] = e^{g_t[c]} sum_r dS[r,c] S_{t-1}[r,c] ;   dS <- dS diag(e^{g_t})
 * The uncentred variant drops the m terms.  States are checkpointed every
 * `seg` tokens and each segment is recomputed forward before its reverse.
 */
int ccq_oracle_gla_fwd_bwd(const ccq_oracle_shape* s, int seg, const double* q, const double* k,
                           const double* v, const double* g, const double* lam,
                           const double* dO, double* o, double* dq, double* dk_out,
                           double* dv_out, double* dg, double* dlam) {
  if (s && s->decay) return 1; /* the decay-aligned statistics: token forward only */
  if (!s || seg <= 0 || s->backbone != 0 || s->t0 != 0 || s->B < 0 || s->T < 0 || s->H < 0 ||
      s->dk <= 0 || s->dv <= 0)
    return 1;
  const int B = s->B, T = s->T, H = s->H, dk = s->dk, dv = s->dv;
  const int nseg = (T + seg - 1) / seg;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    const size_t SZ = (size_t)dv * dk, KZ = (size_t)dk * dk;
    /* checkpoints at each segment start: state before the segment's first token */
    double* ckS = malloc(sizeof(double) * SZ * (nseg > 0 ? nseg : 1));
    double* ckK = malloc(sizeof(double) * KZ * (nseg > 0 ? nseg : 1));
    double* ckm = malloc(sizeof(double) * dk * (nseg > 0 ? nseg : 1));
    /* per-segment recomputation buffers: S_t for t = start-1 .. end-1, K_t, m_t, c_t, qc_t */
    double* segS = malloc(sizeof(double) * SZ * (seg + 1));
    double* segK = malloc(sizeof(double) * KZ * seg);
    double* segm = malloc(sizeof(double) * dk * seg);
    double* segc = malloc(sizeof(double) * dk * seg);
    double* segqc = malloc(sizeof(double) * dk * seg);
    double* S = malloc(sizeof(double) * SZ);
    double* K = malloc(sizeof(double) * KZ);
    double* m = malloc(sizeof(double) * dk);
    double* dS = malloc(sizeof(double) * SZ);
    double* dK = malloc(sizeof(double) * KZ);
    double* dm = malloc(sizeof(double) * dk);
    double* dqc = malloc(sizeof(double) * dk);
    double* dc = malloc(sizeof(double) * dk);
    if (!ckS || !ckK || !ckm || !segS || !segK || !segm || !segc || !segqc || !S || !K || !m ||
        !dS || !dK || !dm || !dqc || !dc) {
#pragma omp atomic write
      err = 2;
    } else {
      memset(S, 0, sizeof(double) * SZ);
      memset(K, 0, sizeof(double) * KZ);
      memset(m, 0, sizeof(double) * dk);
      /* forward sweep: checkpoints and o */
      for (int t = 0; t < T; ++t) {
        if (t % seg == 0) {
          memcpy(ckS + (size_t)(t / seg) * SZ, S, sizeof(double) * SZ);
          memcpy(ckK + (size_t)(t / seg) * KZ, K, sizeof(double) * KZ);
          memcpy(ckm + (size_t)(t / seg) * dk, m, sizeof(double) * dk);
        }
        const size_t ti = tok(s, b, t, h);
        const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv, *gt = g + ti * dk;
        const double tau = t + 1.0;
        for (int a = 0; a < dk; ++a)
          for (int bb = 0; bb < dk; ++bb) K[a * dk + bb] += kt[a] * kt[bb];
        for (int a = 0; a < dk; ++a) m[a] += kt[a];
        double mq = 0.0;
        for (int a = 0; a < dk; ++a) mq += m[a] * qt[a];
        for (int a = 0; a < dk; ++a) {
          double acc = 0.0;
          for (int bb = 0; bb < dk; ++bb) acc += K[a * dk + bb] * qt[bb];
          dqc[a] = qt[a] - lam[ti] * (acc / tau - (s->centered ? m[a] * mq / (tau * tau) : 0.0));
        }
        for (int r = 0; r < dv; ++r)
          for (int a = 0; a < dk; ++a) S[r * dk + a] = S[r * dk + a] * exp(gt[a]) + vt[r] * kt[a];
        for (int r = 0; r < dv; ++r) {
          double acc = 0.0;
          for (int a = 0; a < dk; ++a) acc += S[r * dk + a] * dqc[a];
          o[ti * dv + r] = s->scale * acc;
        }
      }
      memset(dS, 0, sizeof(double) * SZ);
      memset(dK, 0, sizeof(double) * KZ);
      memset(dm, 0, sizeof(double) * dk);
      for (int sg = nseg - 1; sg >= 0; --sg) {
        const int start = sg * seg;
        const int end = (start + seg) < T ? (start + seg) : T;
        /* recompute the segment forward from its checkpoint */
        memcpy(segS, ckS + (size_t)sg * SZ, sizeof(double) * SZ);
        memcpy(K, ckK + (size_t)sg * KZ, sizeof(double) * KZ);
        memcpy(m, ckm + (size_t)sg * dk, sizeof(double) * dk);
        for (int t = start; t < end; ++t) {
          const int lt = t - start;
          const size_t ti = tok(s, b, t, h);
          const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv, *gt = g + ti * dk;
          const double tau = t + 1.0;
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb) K[a * dk + bb] += kt[a] * kt[bb];
          for (int a = 0; a < dk; ++a) m[a] += kt[a];
          memcpy(segK + (size_t)lt * KZ, K, sizeof(double) * KZ);
          memcpy(segm + (size_t)lt * dk, m, sizeof(double) * dk);
          double mq = 0.0;
          for (int a = 0; a < dk; ++a) mq += m[a] * qt[a];
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb) acc += K[a * dk + bb] * qt[bb];
            const double c = acc / tau - (s->centered ? m[a] * mq / (tau * tau) : 0.0);
            segc[(size_t)lt * dk + a] = c;
            segqc[(size_t)lt * dk + a] = qt[a] - lam[ti] * c;
          }
          const double* Sp = segS + (size_t)lt * SZ;
          double* Sn = segS + (size_t)(lt + 1) * SZ;
          for (int r = 0; r < dv; ++r)
            for (int a = 0; a < dk; ++a) Sn[r * dk + a] = Sp[r * dk + a] * exp(gt[a]) + vt[r] * kt[a];
        }
        for (int t = end - 1; t >= start; --t) {
          const int lt = t - start;
          const size_t ti = tok(s, b, t, h);
          const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv, *gt = g + ti * dk;
          const double* dOt = dO + ti * dv;
          const double tau = t + 1.0;
          const double* St = segS + (size_t)(lt + 1) * SZ;
          const double* Sprev = segS + (size_t)lt * SZ;
          const double* Kt = segK + (size_t)lt * KZ;
          const double* mt = segm + (size_t)lt * dk;
          const double* ct = segc + (size_t)lt * dk;
          const double* qct = segqc + (size_t)lt * dk;
          for (int r = 0; r < dv; ++r)
            for (int a = 0; a < dk; ++a) dS[r * dk + a] += s->scale * dOt[r] * qct[a];
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int r = 0; r < dv; ++r) acc += St[r * dk + a] * dOt[r];
            dqc[a] = s->scale * acc;
          }
          double dl = 0.0;
          for (int a = 0; a < dk; ++a) dl -= dqc[a] * ct[a];
          dlam[ti] = dl;
          for (int a = 0; a < dk; ++a) dc[a] = -lam[ti] * dqc[a];
          double mdc = 0.0, mq = 0.0;
          for (int a = 0; a < dk; ++a) { mdc += mt[a] * dc[a]; mq += mt[a] * qt[a]; }
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb) acc += Kt[a * dk + bb] * dc[bb];
            dq[ti * dk + a] = dqc[a] + acc / tau - (s->centered ? mt[a] * mdc / (tau * tau) : 0.0);
          }
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb) dK[a * dk + bb] += dc[a] * qt[bb] / tau;
          if (s->centered)
            for (int a = 0; a < dk; ++a) dm[a] -= (dc[a] * mq + qt[a] * mdc) / (tau * tau);
          for (int r = 0; r < dv; ++r) {
            double acc = 0.0;
            for (int a = 0; a < dk; ++a) acc += dS[r * dk + a] * kt[a];
            dv_out[ti * dv + r] = acc;
          }
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int r = 0; r < dv; ++r) acc += dS[r * dk + a] * vt[r];
            for (int bb = 0; bb < dk; ++bb) acc += (dK[a * dk + bb] + dK[bb * dk + a]) * kt[bb];
            dk_out[ti * dk + a] = acc + dm[a];
          }
          for (int a = 0; a < dk; ++a) {
            const double e = exp(gt[a]);
            double acc = 0.0;
            for (int r = 0; r < dv; ++r) acc += dS[r * dk + a] * Sprev[r * dk + a];
            dg[ti * dk + a] = e * acc;
            for (int r = 0; r < dv; ++r) dS[r * dk + a] *= e;
          }
        }
      }
    }
    free(ckS); free(ckK); free(ckm); free(segS); free(segK); free(segm); free(segc); free(segqc);
    free(S); free(K); free(m); free(dS); free(dK); free(dm); free(dqc); free(dc);
  }
  return err;
}

/*
 * Reverse pass of CCQ-Gated DeltaNet for L = sum_t <dO_t, o_t> (fresh start:
 * zero initial states, t0 = 0).  The contraction part is the one of the GLA
 * reverse pass above; the backbone write is
 *   y_t = S_{t-1} k_t,   S_t = a_t S_{t-1} - a_t b_t y_t k_t^T + b_t v_t k_t^T
 * (a_t = e^{logalpha_t}, b_t = beta_t; the cited Gated DeltaNet recurrence).
 * With dS the adjoint of S_t (after this token's read) and z = dS k_t:
 *   dv_t        = b_t z
 *   dbeta_t     = z . (v_t - a_t y_t)
 *   dlogalpha_t = a_t (<dS, S_{t-1}> - b_t z . y_t)
 *   dk_t       += b_t dS^T (v_t - a_t y_t) - a_t b_t S_{t-1}^T z
 *   dS         <- a_t (dS - b_t z k_t^T)          (adjoint of S_{t-1})
 * States are checkpointed every `seg` tokens and each segment is recomputed
 * forward before its reverse.
 */
int ccq_oracle_gdn_fwd_bwd(const ccq_oracle_shape* s, int seg, const double* q, const double* k,
                           const double* v, const double* logalpha, const double* beta,
                           const double* lam, const double* dO, double* o, double* dq,
                           double* dk_out, double* dv_out, double* dlogalpha, double* dbeta,
                           double* dlam) {
  if (s && s->decay) return 1; /* the decay-aligned statistics: token forward only */
  if (!s || seg <= 0 || s->backbone != 1 || s->t0 != 0 || s->B < 0 || s->T < 0 || s->H < 0 ||
      s->dk <= 0 || s->dv <= 0)
    return 1;
  const int B = s->B, T = s->T, H = s->H, dk = s->dk, dv = s->dv;
  const int nseg = (T + seg - 1) / seg;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    const size_t SZ = (size_t)dv * dk, KZ = (size_t)dk * dk;
    double* ckS = malloc(sizeof(double) * SZ * (nseg > 0 ? nseg : 1));
    double* ckK = malloc(sizeof(double) * KZ * (nseg > 0 ? nseg : 1));
    double* ckm = malloc(sizeof(double) * dk * (nseg > 0 ? nseg : 1));
    double* segS = malloc(sizeof(double) * SZ * (seg + 1));
    double* segK = malloc(sizeof(double) * KZ * seg);
    double* segm = malloc(sizeof(double) * dk * seg);
    double* segc = malloc(sizeof(double) * dk * seg);
    double* segqc = malloc(sizeof(double) * dk * seg);
    double* S = malloc(sizeof(double) * SZ);
    double* K = malloc(sizeof(double) * KZ);
    double* m = malloc(sizeof(double) * dk);
    double* dS = malloc(sizeof(double) * SZ);
    double* dK = malloc(sizeof(double) * KZ);
    double* dm = malloc(sizeof(double) * dk);
    double* dqc = malloc(sizeof(double) * dk);
    double* dc = malloc(sizeof(double) * dk);
    double* y = malloc(sizeof(double) * dv);
    double* z = malloc(sizeof(double) * dv);
    if (!ckS || !ckK || !ckm || !segS || !segK || !segm || !segc || !segqc || !S || !K || !m ||
        !dS || !dK || !dm || !dqc || !dc || !y || !z) {
#pragma omp atomic write
      err = 2;
    } else {
      memset(S, 0, sizeof(double) * SZ);
      memset(K, 0, sizeof(double) * KZ);
      memset(m, 0, sizeof(double) * dk);
      /* forward sweep: checkpoints and o */
      for (int t = 0; t < T; ++t) {
        if (t % seg == 0) {
          memcpy(ckS + (size_t)(t / seg) * SZ, S, sizeof(double) * SZ);
          memcpy(ckK + (size_t)(t / seg) * KZ, K, sizeof(double) * KZ);
          memcpy(ckm + (size_t)(t / seg) * dk, m, sizeof(double) * dk);
        }
        const size_t ti = tok(s, b, t, h);
        const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv;
        const double tau = t + 1.0;
        for (int a = 0; a < dk; ++a)
          for (int bb = 0; bb < dk; ++bb) K[a * dk + bb] += kt[a] * kt[bb];
        for (int a = 0; a < dk; ++a) m[a] += kt[a];
        double mq = 0.0;
        for (int a = 0; a < dk; ++a) mq += m[a] * qt[a];
        for (int a = 0; a < dk; ++a) {
          double acc = 0.0;
          for (int bb = 0; bb < dk; ++bb) acc += K[a * dk + bb] * qt[bb];
          dqc[a] = qt[a] - lam[ti] * (acc / tau - (s->centered ? m[a] * mq / (tau * tau) : 0.0));
        }
        backbone_write(s, S, kt, vt, NULL, logalpha[ti], beta[ti], y);
        for (int r = 0; r < dv; ++r) {
          double acc = 0.0;
          for (int a = 0; a < dk; ++a) acc += S[r * dk + a] * dqc[a];
          o[ti * dv + r] = s->scale * acc;
        }
      }
      memset(dS, 0, sizeof(double) * SZ);
      memset(dK, 0, sizeof(double) * KZ);
      memset(dm, 0, sizeof(double) * dk);
      for (int sg = nseg - 1; sg >= 0; --sg) {
        const int start = sg * seg;
        const int end = (start + seg) < T ? (start + seg) : T;
        memcpy(segS, ckS + (size_t)sg * SZ, sizeof(double) * SZ);
        memcpy(K, ckK + (size_t)sg * KZ, sizeof(double) * KZ);
        memcpy(m, ckm + (size_t)sg * dk, sizeof(double) * dk);
        for (int t = start; t < end; ++t) {
          const int lt = t - start;
          const size_t ti = tok(s, b, t, h);
          const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv;
          const double tau = t + 1.0;
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb) K[a * dk + bb] += kt[a] * kt[bb];
          for (int a = 0; a < dk; ++a) m[a] += kt[a];
          memcpy(segK + (size_t)lt * KZ, K, sizeof(double) * KZ);
          memcpy(segm + (size_t)lt * dk, m, sizeof(double) * dk);
          double mq = 0.0;
          for (int a = 0; a < dk; ++a) mq += m[a] * qt[a];
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb) acc += K[a * dk + bb] * qt[bb];
            const double c = acc / tau - (s->centered ? m[a] * mq / (tau * tau) : 0.0);
            segc[(size_t)lt * dk + a] = c;
            segqc[(size_t)lt * dk + a] = qt[a] - lam[ti] * c;
          }
          double* Sn = segS + (size_t)(lt + 1) * SZ;
          memcpy(Sn, segS + (size_t)lt * SZ, sizeof(double) * SZ);
          backbone_write(s, Sn, kt, vt, NULL, logalpha[ti], beta[ti], y);
        }
        for (int t = end - 1; t >= start; --t) {
          const int lt = t - start;
          const size_t ti = tok(s, b, t, h);
          const double *kt = k + ti * dk, *qt = q + ti * dk, *vt = v + ti * dv;
          const double* dOt = dO + ti * dv;
          const double tau = t + 1.0;
          const double al = exp(logalpha[ti]), bt = beta[ti];
          const double* St = segS + (size_t)(lt + 1) * SZ;
          const double* Sprev = segS + (size_t)lt * SZ;
          const double* Kt = segK + (size_t)lt * KZ;
          const double* mt = segm + (size_t)lt * dk;
          const double* ct = segc + (size_t)lt * dk;
          const double* qct = segqc + (size_t)lt * dk;
          /* read o_t = scale S_t qc_t */
          for (int r = 0; r < dv; ++r)
            for (int a = 0; a < dk; ++a) dS[r * dk + a] += s->scale * dOt[r] * qct[a];
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int r = 0; r < dv; ++r) acc += St[r * dk + a] * dOt[r];
            dqc[a] = s->scale * acc;
          }
          /* contraction qc_t = q_t - lam_t c_t */
          double dl = 0.0;
          for (int a = 0; a < dk; ++a) dl -= dqc[a] * ct[a];
          dlam[ti] = dl;
          for (int a = 0; a < dk; ++a) dc[a] = -lam[ti] * dqc[a];
          double mdc = 0.0, mq = 0.0;
          for (int a = 0; a < dk; ++a) { mdc += mt[a] * dc[a]; mq += mt[a] * qt[a]; }
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int bb = 0; bb < dk; ++bb) acc += Kt[a * dk + bb] * dc[bb];
            dq[ti * dk + a] = dqc[a] + acc / tau - (s->centered ? mt[a] * mdc / (tau * tau) : 0.0);
          }
          for (int a = 0; a < dk; ++a)
            for (int bb = 0; bb < dk; ++bb) dK[a * dk + bb] += dc[a] * qt[bb] / tau;
          if (s->centered)
            for (int a = 0; a < dk; ++a) dm[a] -= (dc[a] * mq + qt[a] * mdc) / (tau * tau);
          /* backbone write */
          for (int r = 0; r < dv; ++r) {
            double ay = 0.0, az = 0.0;
            for (int a = 0; a < dk; ++a) {
              ay += Sprev[r * dk + a] * kt[a];
              az += dS[r * dk + a] * kt[a];
            }
            y[r] = ay;
            z[r] = az;
          }
          double db = 0.0, zy = 0.0, dSS = 0.0;
          for (int r = 0; r < dv; ++r) {
            dv_out[ti * dv + r] = bt * z[r];
            db += z[r] * (vt[r] - al * y[r]);
            zy += z[r] * y[r];
          }
          for (size_t i = 0; i < SZ; ++i) dSS += dS[i] * Sprev[i];
          dbeta[ti] = db;
          dlogalpha[ti] = al * (dSS - bt * zy);
          for (int a = 0; a < dk; ++a) {
            double acc = 0.0;
            for (int r = 0; r < dv; ++r)
              acc += bt * dS[r * dk + a] * (vt[r] - al * y[r]) - al * bt * Sprev[r * dk + a] * z[r];
            for (int bb = 0; bb < dk; ++bb) acc += (dK[a * dk + bb] + dK[bb * dk + a]) * kt[bb];
            dk_out[ti * dk + a] = acc + dm[a];
          }
          for (int r = 0; r < dv; ++r)
            for (int a = 0; a < dk; ++a) dS[r * dk + a] = al * (dS[r * dk + a] - bt * z[r] * kt[a]);
        }
      }
    }
    free(ckS); free(ckK); free(ckm); free(segS); free(segK); free(segm); free(segc); free(segqc);
    free(S); free(K); free(m); free(dS); free(dK); free(dm); free(dqc); free(dc); free(y); free(z);
  }
  return err;
}

/*
 * Pre-processing of one layer's raw queries and keys (Alg. 1, the per-chunk
 * normalisation and gate lines; Eq. clean for the gate):
 *   qbar = q / max(|q|, 1e-12), kbar = k / max(|k|, 1e-12)   per head;
 *   lambda[h] = sigmoid(sum_j W[h][j] qraw[j] + b[h]),
 * where qraw is the token's query before the split into heads (all H*dk
 * features, head-major) and W is [H, H*dk].  Layouts: q, k [B,T,H,dk];
 * lambda [B,T,H].  Outputs may alias nothing.
 */
int ccq_oracle_prep(int32_t B, int32_t T, int32_t H, int32_t dk, const double* q, const double* k,
                    const double* W, const double* bias, double* qbar, double* kbar, double* lam) {
  if (B < 0 || T < 0 || H <= 0 || dk <= 0) return 1;
  const int64_t ntok = (int64_t)B * T;
  const int64_t E = (int64_t)H * dk;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < ntok; ++t) {
    const double* qr = q + t * E;
    const double* kr = k + t * E;
    for (int h = 0; h < H; ++h) {
      double qq = 0.0, kk = 0.0;
      for (int c = 0; c < dk; ++c) {
        qq += qr[h * dk + c] * qr[h * dk + c];
        kk += kr[h * dk + c] * kr[h * dk + c];
      }
      const double qn = sqrt(qq) > 1e-12 ? sqrt(qq) : 1e-12;
      const double kn = sqrt(kk) > 1e-12 ? sqrt(kk) : 1e-12;
      for (int c = 0; c < dk; ++c) {
        qbar[t * E + h * dk + c] = qr[h * dk + c] / qn;
        kbar[t * E + h * dk + c] = kr[h * dk + c] / kn;
      }
      double z = bias[h];
      for (int64_t j = 0; j < E; ++j) z += W[h * E + j] * qr[j];
      lam[t * H + h] = 1.0 / (1.0 + exp(-z));
    }
  }
  return 0;
}
