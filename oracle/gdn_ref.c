/*
 * gdn_ref.c -- CPU oracle for the Gated DeltaNet recurrence (fp64).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing on the product path may link, load or call
 * this file; only the test suite, the smoke check and the CPU-baseline leg of
 * the benchmark use it. It shares no code, header or constant with the HIP
 * library.
 *
 * What it computes (the plain definition, token by token, in double precision):
 * the gated delta rule of the paper's Section 3.2 ("Kernel Techniques", the
 * display equations for old_v, delta and S'). Per token t of one sequence and
 * one value head h, with the state S stored as a d_v x d_k matrix (row v holds
 * the d_k key coefficients of value channel v):
 *
 *     alpha = exp(g_t)                      g_t is the LOG of the paper's gate
 *     S     <- alpha * S                    pre-scaled state ("gS")
 *     old   =  S k_t                        old_v = k^T (gS), one entry per row
 *     delta =  beta_t * (v_t - old)         delta = beta (v - old_v)
 *     S     <- S + delta k_t^T              S' = gS + k delta^T (transposed store)
 *     o_t   =  S q_t                        output read from the UPDATED state
 *
 * which is S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
 * o_t = S_t q_t. The paper also rewrites the output as q^T(gS) + delta (q^T k);
 * the oracle deliberately evaluates the definition (a dot product against the
 * updated state) and the test suite checks the rewrite against it.
 *
 * Grouped heads: value head h reads query/key head h / (HV / HQK), i.e.
 * consecutive value heads share one key head.
 *
 * Layouts (all row-major, contiguous, double):
 *   q, k          [T_total, HQK, DK]
 *   v             [T_total, HV, DV]
 *   g, beta       [T_total, HV]
 *   cu_seqlens    [N + 1] int32, cu[0] = 0, non-decreasing, cu[N] = T_total
 *   s0, s_final   [N, HV, DV, DK]  (s0 may be NULL for a zero initial state)
 *   o             [T_total, HV, DV]
 *
 * Work is split over (sequence, value head) chains with OpenMP; every chain is
 * an independent token-serial loop, so the result does not depend on the
 * number of threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* One token of the recurrence on one (sequence, value head) chain. */
static void ref_token_step(double *S, const double *q, const double *k,
                           const double *v, double g, double beta, double *o,
                           int dk, int dv) {
  const double alpha = exp(g);
  for (int r = 0; r < dv; ++r) {
    double *row = S + (size_t)r * dk;
    double old = 0.0;
    for (int c = 0; c < dk; ++c) {
      row[c] *= alpha;
      old += row[c] * k[c];
    }
    const double delta = beta * (v[r] - old);
    double out = 0.0;
    for (int c = 0; c < dk; ++c) {
      row[c] += delta * k[c];
      out += row[c] * q[c];
    }
    o[r] = out;
  }
}

/* Returns 0 on success, a negative value on a malformed argument. */
int gdn_ref_prefill(const double *q, const double *k, const double *v,
                    const double *g, const double *beta,
                    const int32_t *cu_seqlens, const double *s0, double *o,
                    double *s_final, int32_t n_seqs, int64_t n_tokens,
                    int32_t hqk, int32_t hv, int32_t dk, int32_t dv) {
  if (n_seqs < 0 || n_tokens < 0 || hqk <= 0 || hv <= 0 || dk <= 0 || dv <= 0)
    return -1;
  if (hv % hqk != 0) return -2;
  if (!cu_seqlens || !s_final) return -3;
  if (cu_seqlens[0] != 0 || cu_seqlens[n_seqs] != n_tokens) return -4;
  for (int32_t n = 0; n < n_seqs; ++n)
    if (cu_seqlens[n + 1] < cu_seqlens[n]) return -5;
  const int32_t group = hv / hqk;
  const size_t sdim = (size_t)dv * dk;
  const int64_t chains = (int64_t)n_seqs * hv;

#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t ch = 0; ch < chains; ++ch) {
    const int32_t n = (int32_t)(ch / hv);
    const int32_t h = (int32_t)(ch % hv);
    const int32_t hk = h / group;
    double *S = s_final + (size_t)ch * sdim;
    if (s0)
      memmove(S, s0 + (size_t)ch * sdim, sdim * sizeof(double));
    else
      memset(S, 0, sdim * sizeof(double));
    for (int64_t t = cu_seqlens[n]; t < cu_seqlens[n + 1]; ++t) {
      ref_token_step(S, q + ((size_t)t * hqk + hk) * dk,
                     k + ((size_t)t * hqk + hk) * dk,
                     v + ((size_t)t * hv + h) * dv, g[(size_t)t * hv + h],
                     beta[(size_t)t * hv + h], o + ((size_t)t * hv + h) * dv,
                     dk, dv);
    }
  }
  return 0;
}

/* One decode step: every batch entry is a sequence of exactly one token, and
 * state [B, HV, DV, DK] is advanced in place. */
int gdn_ref_decode(const double *q, const double *k, const double *v,
                   const double *g, const double *beta, double *state,
                   double *o, int32_t batch, int32_t hqk, int32_t hv,
                   int32_t dk, int32_t dv) {
  if (batch < 0 || hqk <= 0 || hv <= 0 || dk <= 0 || dv <= 0) return -1;
  if (hv % hqk != 0) return -2;
  if (!state) return -3;
  const int32_t group = hv / hqk;
  const size_t sdim = (size_t)dv * dk;
  const int64_t chains = (int64_t)batch * hv;

#pragma omp parallel for schedule(static)
  for (int64_t ch = 0; ch < chains; ++ch) {
    const int32_t b = (int32_t)(ch / hv);
    const int32_t h = (int32_t)(ch % hv);
    const int32_t hk = h / group;
    ref_token_step(state + (size_t)ch * sdim, q + ((size_t)b * hqk + hk) * dk,
                   k + ((size_t)b * hqk + hk) * dk,
                   v + ((size_t)b * hv + h) * dv, g[ch], beta[ch],
                   o + ((size_t)b * hv + h) * dv, dk, dv);
  }
  return 0;
}

/*
 * Gate activation (paper, Section 3.2, the first two display lines of the
 * one-pass form): the paper's multiplicative gate is
 * exp(-exp(A_log) * softplus(a + b_dt)) and beta = sigma(b). The oracle's
 * recurrence takes the LOG of that gate, so per token t and value head h
 *
 *     g[t, h]    = -exp(A_log[h]) * softplus(a[t, h] + dt_bias[h])
 *     beta[t, h] = 1 / (1 + exp(-b[t, h]))
 *
 * with softplus(x) = log(1 + exp(x)), evaluated as x + log1p(exp(-x)) for
 * x > 0 so that exp never overflows. a, b, g, beta: [T, HV]; A_log, dt_bias:
 * [HV].
 */
static double ref_softplus(double x) {
  return x > 0.0 ? x + log1p(exp(-x)) : log1p(exp(x));
}

int gdn_ref_gate(const double *a, const double *b, const double *A_log,
                 const double *dt_bias, double *g, double *beta,
                 int64_t n_tokens, int32_t hv) {
  if (n_tokens < 0 || hv <= 0) return -1;
  for (int64_t t = 0; t < n_tokens; ++t) {
    for (int32_t h = 0; h < hv; ++h) {
      const size_t i = (size_t)t * hv + h;
      g[i] = -exp(A_log[h]) * ref_softplus(a[i] + dt_bias[h]);
      beta[i] = 1.0 / (1.0 + exp(-b[i]));
    }
  }
  return 0;
}

int gdn_ref_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
