/*
 * oracle.c -- plain fp64 CPU reference for delta-rule linear-attention prefill.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness oracle: only the
 * test suite, the smoke check and the CPU-baseline leg of the benchmark may
 * load or call it.  The GPU library shares no code, header, table or build
 * step with it, and the product path never routes through it.
 *
 * What it computes (paper, Sec. 2.1 "Architecture of Linear-Attention
 * Hybrids"): per head, a fixed-size recurrent state is updated once per token
 * from k_t and v_t, and the token's output is then read from the UPDATED
 * state with q_t.  The update is the gated delta rule of Gated DeltaNet (the
 * GDN layer the paper evaluates, Sec. 2.1 and Sec. 7.1 "Models and
 * Datasets"), written with the state S (d_v x d_k):
 *
 *     S_t = alpha_t * S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = scale * S_t q_t
 *
 * KDA (Kimi Delta Attention, the paper's second mechanism, Sec. 7.1) replaces
 * the scalar alpha_t by a per-key-channel decay vector applied on the key
 * side of S before the delta update:
 *
 *     S_t = S_{t-1} Diag(alpha_t) (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *
 * Storage convention: the oracle keeps H = S^T (d_k rows, d_v columns, row =
 * key channel), the same orientation as the library's s0 / s_final buffers.
 * In that orientation one token step is, exactly equivalent to the formulas
 * above:
 *
 *     H <- Diag(a_t) H                (a_t = exp(g_t); scalar for GDN)
 *     p <- H^T k_t
 *     u <- beta_t (v_t - p)
 *     H <- H + k_t u^T
 *     o_t <- scale * H^T q_t
 *
 * Gates enter as log-gates g (alpha = exp(g)), the form in which the paper's
 * kernels keep gates in FP32 (Sec. 7.1 "Baselines": FP32 gates/states).
 *
 * Everything is fp64.  Inputs are the exact values the GPU consumed (bf16 or
 * fp32 values widened to fp64 by the caller).  The chunkwise Map-Reduce-Map
 * decomposition the GPU uses (Sec. 2.1 "Chunkwise Map-Reduce-Map Execution")
 * reaches this same result up to rounding; this file deliberately does no
 * chunking, blocking or reordering.
 *
 * Varlen packing: sequences are packed token-major and delimited by
 * cu_seqlens[0..N] (cu_seqlens[0] = 0, cu_seqlens[N] = T_total).  Grouped
 * heads: value head h reads query/key head h / (Hv / Hqk).
 *
 * Layouts (row-major, fp64):
 *   q, k   [T_total, Hqk, Dk]      v, o [T_total, Hv, Dv]
 *   g      GDN [T_total, Hv]       KDA [T_total, Hv, Dk]
 *   beta   [T_total, Hv]
 *   s0, s_final  [N, Hv, Dk, Dv]   (s0 may be NULL: zero initial state)
 *
 * Returns 0 on success, -1 on an invalid argument (nothing written).
 */
#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int oracle_check(const int *cu, int N, int T_total, int Hqk, int Hv,
                        int Dk, int Dv) {
  if (N < 1 || T_total < 0 || Hqk < 1 || Hv < 1 || Dk < 1 || Dv < 1)
    return -1;
  if (Hv % Hqk != 0) return -1;
  if (cu[0] != 0 || cu[N] != T_total) return -1;
  for (int n = 0; n < N; ++n)
    if (cu[n + 1] < cu[n]) return -1;
  return 0;
}

/* One (sequence, value head) pair: the token loop of the definition above. */
static void oracle_one_head(int kda, const double *q, const double *k,
                            const double *v, const double *g,
                            const double *beta, const double *s0_nh,
                            int t_begin, int t_end, int h, int Hqk, int Hv,
                            int Dk, int Dv, double scale, double *o,
                            double *sfin_nh, double *H, double *p) {
  const int group = Hv / Hqk;
  const int hk = h / group;
  if (s0_nh)
    memcpy(H, s0_nh, sizeof(double) * (size_t)Dk * Dv);
  else
    memset(H, 0, sizeof(double) * (size_t)Dk * Dv);

  for (int t = t_begin; t < t_end; ++t) {
    const double *kt = k + ((size_t)t * Hqk + hk) * Dk;
    const double *qt = q + ((size_t)t * Hqk + hk) * Dk;
    const double *vt = v + ((size_t)t * Hv + h) * Dv;
    const double bt = beta[(size_t)t * Hv + h];

    /* decay: H <- Diag(a_t) H */
    if (kda) {
      const double *gt = g + ((size_t)t * Hv + h) * Dk;
      for (int i = 0; i < Dk; ++i) {
        const double a = exp(gt[i]);
        for (int j = 0; j < Dv; ++j) H[(size_t)i * Dv + j] *= a;
      }
    } else {
      const double a = exp(g[(size_t)t * Hv + h]);
      for (size_t e = 0; e < (size_t)Dk * Dv; ++e) H[e] *= a;
    }

    /* p <- H^T k_t */
    for (int j = 0; j < Dv; ++j) p[j] = 0.0;
    for (int i = 0; i < Dk; ++i) {
      const double ki = kt[i];
      for (int j = 0; j < Dv; ++j) p[j] += H[(size_t)i * Dv + j] * ki;
    }
    /* u <- beta_t (v_t - p) (stored over p) */
    for (int j = 0; j < Dv; ++j) p[j] = bt * (vt[j] - p[j]);
    /* H <- H + k_t u^T */
    for (int i = 0; i < Dk; ++i) {
      const double ki = kt[i];
      for (int j = 0; j < Dv; ++j) H[(size_t)i * Dv + j] += ki * p[j];
    }
    /* o_t <- scale * H^T q_t, from the updated state */
    double *ot = o + ((size_t)t * Hv + h) * Dv;
    for (int j = 0; j < Dv; ++j) ot[j] = 0.0;
    for (int i = 0; i < Dk; ++i) {
      const double qi = qt[i];
      for (int j = 0; j < Dv; ++j) ot[j] += H[(size_t)i * Dv + j] * qi;
    }
    for (int j = 0; j < Dv; ++j) ot[j] *= scale;
  }
  if (sfin_nh) memcpy(sfin_nh, H, sizeof(double) * (size_t)Dk * Dv);
}

static int oracle_run(int kda, const double *q, const double *k,
                      const double *v, const double *g, const double *beta,
                      const double *s0, const int *cu_seqlens, int N,
                      int T_total, int Hqk, int Hv, int Dk, int Dv,
                      double scale, double *o, double *s_final,
                      int nthreads) {
  if (!q || !k || !v || !g || !beta || !cu_seqlens || !o) return -1;
  if (oracle_check(cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv)) return -1;
  const long pairs = (long)N * Hv;
  int bad = 0;
#ifdef _OPENMP
  if (nthreads < 1) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads) reduction(| : bad)
#endif
  {
    double *H = (double *)malloc(sizeof(double) * (size_t)Dk * Dv);
    double *p = (double *)malloc(sizeof(double) * (size_t)Dv);
    if (!H || !p) {
      bad = 1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (long pr = 0; pr < pairs; ++pr) {
        const int n = (int)(pr / Hv), h = (int)(pr % Hv);
        const size_t st = ((size_t)n * Hv + h) * Dk * Dv;
        oracle_one_head(kda, q, k, v, g, beta, s0 ? s0 + st : NULL,
                        cu_seqlens[n], cu_seqlens[n + 1], h, Hqk, Hv, Dk, Dv,
                        scale, o, s_final ? s_final + st : NULL, H, p);
      }
    }
    free(H);
    free(p);
  }
  (void)nthreads;
  return bad ? -1 : 0;
}

/* Gated DeltaNet: scalar log-gate g[T_total, Hv]. */
int oracle_gdn_prefill(const double *q, const double *k, const double *v,
                       const double *g, const double *beta, const double *s0,
                       const int *cu_seqlens, int N, int T_total, int Hqk,
                       int Hv, int Dk, int Dv, double scale, double *o,
                       double *s_final, int nthreads) {
  return oracle_run(0, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv,
                    Dk, Dv, scale, o, s_final, nthreads);
}

/* KDA: per-key-channel log-gate g[T_total, Hv, Dk]. */
int oracle_kda_prefill(const double *q, const double *k, const double *v,
                       const double *g, const double *beta, const double *s0,
                       const int *cu_seqlens, int N, int T_total, int Hqk,
                       int Hv, int Dk, int Dv, double scale, double *o,
                       double *s_final, int nthreads) {
  return oracle_run(1, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv,
                    Dk, Dv, scale, o, s_final, nthreads);
}

/*
 * Preprocessing of raw projections, the step in front of the recurrence.
 * The paper accelerates the layer's projections around the LA core by
 * operator fusion (Sec. 7, "Implementation and Evaluation", full-layer
 * implementation); the elementwise maps that turn projections into the
 * recurrence's inputs are the ones its workloads use (per-token L2
 * normalisation of q and k, a softplus log-gate and a sigmoid write strength).
 * In place, fp64, one token at a time:
 *
 *   flag 1  q_t <- q_t / max(||q_t||_2, 1e-6) and the same for k_t, per token
 *           and query/key head
 *   flag 2  g <- -softplus(g) = -log(1 + e^g), every element (GDN [T, Hv],
 *           KDA [T, Hv, Dk])
 *   flag 4  beta <- 1 / (1 + e^-beta)
 *
 * softplus is evaluated as max(x, 0) + log1p(e^-|x|), which is log(1 + e^x)
 * rearranged so that the exponential never overflows.
 * Returns 0, or -1 on an invalid argument (nothing changed).
 */
int oracle_preprocess(double *q, double *k, double *g, double *beta, int T,
                      int Hqk, int Hv, int Dk, int kda, int flags) {
  if (T < 0 || Hqk < 1 || Hv < 1 || Dk < 1 || (flags & ~7)) return -1;
  if (T == 0) return 0;
  if (!q || !k || !g || !beta) return -1;
  if (flags & 1) {
    for (size_t r = 0; r < (size_t)T * Hqk; ++r) {
      double *rows[2] = {q + r * Dk, k + r * Dk};
      for (int w = 0; w < 2; ++w) {
        double ss = 0.0;
        for (int i = 0; i < Dk; ++i) ss += rows[w][i] * rows[w][i];
        double nrm = sqrt(ss);
        if (nrm < 1e-6) nrm = 1e-6;
        for (int i = 0; i < Dk; ++i) rows[w][i] /= nrm;
      }
    }
  }
  if (flags & 2) {
    const size_t n = (size_t)T * Hv * (kda ? Dk : 1);
    for (size_t e = 0; e < n; ++e) {
      const double x = g[e];
      g[e] = -((x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x))));
    }
  }
  if (flags & 4) {
    for (size_t e = 0; e < (size_t)T * Hv; ++e) beta[e] = 1.0 / (1.0 + exp(-beta[e]));
  }
  return 0;
}
