/*
 * dla_oracle.c -- plain float64 CPU oracle of the Dynamic Linear Attention (DLA)
 * layer forward (arXiv 2606.10650).
 *
 * TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code with
 * the HIP path: no headers, no helpers, no tables.
 *
 * The method is an online heuristic, so the oracle is the algorithm itself, run
 * token by token per head in float64, in the order the paper states it:
 *
 *   for every token t:
 *     every cached state decays by alpha_t = exp(g_t)            (reading U2)
 *     token state s_t = k_t v_t^T  (identity feature map, Sec. 2.1)
 *     State Information Score against the newest state S (eq. importance_score,
 *     with RMSNorm applied to both states, Sec. 3.1):
 *         I_t = || N(s_t) - N(S) ||_F / ( || N(S) ||_F + eps )
 *         N(X) = X / sqrt( sum(X^2) / (dk dv) + eps_rms )
 *     boundary b_t = [I_t >= tau]                                 (Sec. 3.1)
 *     b_t = 0: accumulate s_t into the newest state;
 *     b_t = 1: if the cache holds C states, merge the adjacent pair of lowest
 *              information density argmin_i (I_i + I_{i+1}) / (n_i + n_{i+1})
 *              (Alg. 2, Sec. 3.2), then append s_t as a new state.
 *     readout o_t = sum_j lambda_{t,j} S_j^T q_t     (eq. capacity_bounded_output)
 *
 * With a step size beta_t (the Gated DeltaNet form of the base model, Sec. 2.2,
 * eq. delta_rule_rnn, in this orientation S = sum k v^T, o = S^T q), the newest
 * state follows the delta rule while it accumulates, and a token writes
 * beta_t s_t:
 *     b_t = 0: S <- (I - beta_t k_t k_t^T) S + beta_t s_t   (S already decayed)
 *     b_t = 1: the new state is beta_t s_t
 * Closed states only decay.  The score still compares s_t with the newest state
 * before this token's update (it is scale-invariant, so beta does not enter it).
 *
 * Readings where the paper is silent or inconsistent (each one is listed with
 * its reasons in the design notes of the repository):
 *   - the score compares the RMS-normalised token state with the RMS-normalised
 *     newest state (Alg. 1 and eq. importance_score agree when the equation's
 *     S_t is the token state);
 *   - Alg. 1 both merges s_t and appends it when I_t >= tau; the update rule of
 *     Sec. 3.1 is exclusive (accumulate OR open), which is what is done here;
 *   - the first token of an empty cache opens a state with score 0;
 *   - a new state's aggregated score includes its first token's score;
 *   - the capacity merge happens only when a new state is opened and the cache
 *     is full; the just-closed state is a candidate, the new one is not;
 *   - C = 1 forces b_t = 0 after the first token (no adjacent pair exists);
 *   - argmin ties go to the lowest index;
 *   - lambda is indexed by the chronological position (0 = oldest) of a state
 *     in the cache after token t is absorbed; NULL lambda means 1;
 *   - token counts and aggregated scores do not decay.
 *
 * "full" mode keeps every state as a matrix and produces outputs and the final
 * cache.  "decisions" mode runs Alg. 1 on the newest state only and Alg. 2 on
 * the scalar (n, I) pairs; it yields the same boundaries, scores and merge
 * indices because a capacity merge never involves the state that receives the
 * next tokens, and skips everything else.  The two modes are compared by the
 * test-suite.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_BAD_MERGE_OVERRIDE 1
#define ORACLE_BAD_ARG 2
#define ORACLE_NOMEM 3

int dla_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Frobenius norm of an array of n doubles. */
static double frob(const double* x, int64_t n) {
  double acc = 0.0;
  for (int64_t i = 0; i < n; ++i) acc += x[i] * x[i];
  return sqrt(acc);
}

/* Delta-rule erase of a d_k x d_v state: S <- (I - beta k k^T) S, through
 * u = S^T k (work: dv doubles). */
static void delta_erase(double* S, const double* k, double beta, int32_t dk, int32_t dv,
                        double* u) {
  for (int32_t c = 0; c < dv; ++c) u[c] = 0.0;
  for (int32_t a = 0; a < dk; ++a)
    for (int32_t c = 0; c < dv; ++c) u[c] += k[a] * S[a * dv + c];
  for (int32_t a = 0; a < dk; ++a)
    for (int32_t c = 0; c < dv; ++c) S[a * dv + c] -= beta * k[a] * u[c];
}

/* State Information Score of token state s against state S (both D values),
 * with RMSNorm (unit weight, over the whole flattened state) on both. */
static double info_score(const double* s, const double* S, int64_t D, double eps,
                         double eps_rms, double* ns, double* nS) {
  double ss = 0.0, SS = 0.0;
  for (int64_t i = 0; i < D; ++i) {
    ss += s[i] * s[i];
    SS += S[i] * S[i];
  }
  const double rs = sqrt(ss / (double)D + eps_rms);
  const double rS = sqrt(SS / (double)D + eps_rms);
  for (int64_t i = 0; i < D; ++i) {
    ns[i] = s[i] / rs;
    nS[i] = S[i] / rS;
  }
  double dd = 0.0;
  for (int64_t i = 0; i < D; ++i) {
    const double d = ns[i] - nS[i];
    dd += d * d;
  }
  return sqrt(dd) / (frob(nS, D) + eps);
}

static int run_head(int64_t T, int32_t C, int32_t dk, int32_t dv, const double* q,
                    const double* k, const double* v, const double* g, const double* beta,
                    const double* lam, double tau, double eps, double eps_rms, const int8_t* b_ovr,
                    const int32_t* m_ovr, int32_t full, double* out, int8_t* b_out,
                    int32_t* merge_out, double* score_out, int32_t* m_out, double* margin_b,
                    double* margin_m, double* mag_out, double* u_out, int32_t* cache_m,
                    int64_t* n, double* ibar, double* S) {
  const int64_t D = (int64_t)dk * dv;
  double* s = (double*)malloc(sizeof(double) * (D * 3 + dv));
  double* dens = (double*)malloc(sizeof(double) * (C > 1 ? C : 1));
  if (!s || !dens) {
    free(s);
    free(dens);
    return ORACLE_NOMEM;
  }
  double* y = s + 3 * D;
  double* ns = s + D;
  double* nS = s + 2 * D;
  int32_t m = *cache_m;
  int rc = ORACLE_OK;

  for (int64_t t = 0; t < T; ++t) {
    const double* kt = k + t * dk;
    const double* vt = v + t * dv;
    const double alpha = exp(g[t]);

    /* every cached state decays (decisions mode tracks only the newest) */
    for (int32_t j = full ? 0 : (m > 0 ? m - 1 : 0); j < m; ++j)
      for (int64_t i = 0; i < D; ++i) S[j * D + i] *= alpha;

    /* token state s_t = k_t v_t^T */
    for (int32_t a = 0; a < dk; ++a)
      for (int32_t c = 0; c < dv; ++c) s[a * dv + c] = kt[a] * vt[c];

    double I = 0.0;
    int b;
    int free_b = 0;
    if (m == 0) {
      b = 1; /* first token of an empty cache */
    } else {
      I = info_score(s, S + (int64_t)(m - 1) * D, D, eps, eps_rms, ns, nS);
      b = (I >= tau) ? 1 : 0;
      free_b = 1;
      if (b_ovr && b_ovr[t] != -1) {
        b = b_ovr[t] ? 1 : 0;
        free_b = 0;
      }
      if (C == 1) {
        b = 0;
        free_b = 0;
      }
    }

    /* the token's write (the score above used the unscaled token state) */
    if (beta)
      for (int64_t i = 0; i < D; ++i) s[i] *= beta[t];

    int32_t merged = -1;
    double mgap = INFINITY;
    if (!b) {
      double* So = S + (int64_t)(m - 1) * D;
      if (beta) delta_erase(So, kt, beta[t], dk, dv, y);
      for (int64_t i = 0; i < D; ++i) So[i] += s[i];
      n[m - 1] += 1;
      ibar[m - 1] += I;
      /* the newest state took k_t u_t^T: u_t = beta_t (v_t - y), y the
       * decayed state's S^T k_t (with no beta, u_t = v_t) */
      if (u_out)
        for (int32_t c = 0; c < dv; ++c)
          u_out[t * dv + c] = beta ? beta[t] * (vt[c] - y[c]) : vt[c];
    } else {
      /* the new state is k_t u_t^T with u_t = beta_t v_t (or v_t) */
      if (u_out)
        for (int32_t c = 0; c < dv; ++c) u_out[t * dv + c] = beta ? beta[t] * vt[c] : vt[c];
      if (m == C) {
        /* Alg. 2: lowest-density adjacent pair among the C cached states */
        int32_t best = 0;
        for (int32_t i = 0; i + 1 < C; ++i) {
          dens[i] = (ibar[i] + ibar[i + 1]) / (double)(n[i] + n[i + 1]);
          if (dens[i] < dens[best]) best = i;
        }
        double second = INFINITY;
        for (int32_t i = 0; i + 1 < C; ++i)
          if (i != best && dens[i] < second) second = dens[i];
        if (m_ovr && m_ovr[t] != -1) {
          if (m_ovr[t] < 0 || m_ovr[t] > C - 2) {
            rc = ORACLE_BAD_MERGE_OVERRIDE;
            break;
          }
          best = m_ovr[t];
        } else if (C > 2) {
          const double d1 = dens[best];
          mgap = (second - d1) / (fabs(d1) > 0.0 ? fabs(d1) : 1e-300);
        }
        /* S_i* <- S_i* + S_i*+1 ; n, I summed ; later states shift down */
        if (full)
          for (int64_t i = 0; i < D; ++i) S[best * D + i] += S[(best + 1) * D + i];
        n[best] += n[best + 1];
        ibar[best] += ibar[best + 1];
        for (int32_t j = best + 1; j + 1 < m; ++j) {
          if (full) memcpy(S + j * D, S + (j + 1) * D, sizeof(double) * D);
          n[j] = n[j + 1];
          ibar[j] = ibar[j + 1];
        }
        m -= 1;
        merged = best;
      }
      memcpy(S + (int64_t)m * D, s, sizeof(double) * D);
      n[m] = 1;
      ibar[m] = I;
      m += 1;
    }

    if (out) {
      /* o_t = sum_j lambda_{t,j} S_j^T q_t, one term y_j = S_j^T q_t per state.
       * mag_t = sum_j |lambda_{t,j}| ||S_j||_F ||q_t|| bounds the sizes of the
       * terms the sum adds up (||y_j|| <= ||S_j||_F ||q_t||); it is the scale
       * against which a perturbation of the stored states is measured. */
      double* ot = out + t * dv;
      const double* qt = q + t * dk;
      double mag = 0.0;
      for (int32_t c = 0; c < dv; ++c) ot[c] = 0.0;
      for (int32_t j = 0; j < m; ++j) {
        const double lj = lam ? lam[t * C + j] : 1.0;
        const double* Sj = S + (int64_t)j * D;
        for (int32_t c = 0; c < dv; ++c) y[c] = 0.0;
        for (int32_t a = 0; a < dk; ++a)
          for (int32_t c = 0; c < dv; ++c) y[c] += qt[a] * Sj[a * dv + c];
        for (int32_t c = 0; c < dv; ++c) ot[c] += lj * y[c];
        if (mag_out) mag += fabs(lj) * frob(Sj, D);
      }
      if (mag_out) mag_out[t] = mag * frob(qt, dk);
    }
    if (b_out) b_out[t] = (int8_t)b;
    if (merge_out) merge_out[t] = merged;
    if (score_out) score_out[t] = I;
    if (m_out) m_out[t] = m;
    if (margin_b) margin_b[t] = free_b ? fabs(I - tau) : INFINITY;
    if (margin_m) margin_m[t] = mgap;
  }
  *cache_m = m;
  free(s);
  free(dens);
  return rc;
}

/*
 * Run the layer forward over n_heads independent heads of T tokens.
 *
 * Layouts (row-major): q, k [n_heads][T][dk]; v [n_heads][T][dv]; g [n_heads][T];
 * beta [n_heads][T] or NULL (NULL: no delta rule, a token writes s_t);
 * lam [n_heads][T][C] or NULL; overrides [n_heads][T] or NULL (-1 = free);
 * outputs out [n_heads][T][dv]; b_out, merge_out, score_out, m_out, margin_b,
 * margin_m, mag_out [n_heads][T]; u_out [n_heads][T][dv], the vector u_t with
 * which the token's write is k_t u_t^T (beta_t (v_t - S^T k_t) joining, beta_t
 * v_t opening; v_t without beta); each output may be NULL (mag_out is written
 * only with out).
 *
 * The cache is read and written: cache_m [n_heads], cache_n and cache_ibar
 * [n_heads][C], cache_S [n_heads][C][dk][dv] -- chronological order, true
 * (decayed) states at the last absorbed token.  An empty cache has m = 0.
 * In decisions mode (full == 0) only state m-1 of cache_S is meaningful.
 *
 * Returns 0, or ORACLE_BAD_MERGE_OVERRIDE if a forced merge index is outside
 * [0, C-2] for some head.
 */
int dla_oracle_forward(int64_t n_heads, int64_t T, int32_t C, int32_t dk, int32_t dv,
                       const double* q, const double* k, const double* v, const double* g,
                       const double* beta, const double* lam, double tau, double eps,
                       double eps_rms, const int8_t* b_ovr, const int32_t* m_ovr, int32_t full,
                       double* out,
                       int8_t* b_out, int32_t* merge_out, double* score_out, int32_t* m_out,
                       double* margin_b, double* margin_m, double* mag_out, double* u_out,
                       int32_t* cache_m, int64_t* cache_n, double* cache_ibar,
                       double* cache_S) {
  if (n_heads < 0 || T < 0 || C < 1 || dk < 1 || dv < 1 || !k || !v || !g || !cache_m ||
      !cache_n || !cache_ibar || !cache_S)
    return ORACLE_BAD_ARG;
  if (out && (!q || !full)) return ORACLE_BAD_ARG;
  const int64_t D = (int64_t)dk * dv;
  int rc = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t h = 0; h < n_heads; ++h) {
    const int64_t tok = h * T;
    int r = run_head(T, C, dk, dv, q ? q + tok * dk : NULL, k + tok * dk, v + tok * dv, g + tok,
                     beta ? beta + tok : NULL, lam ? lam + tok * C : NULL, tau, eps, eps_rms, b_ovr ? b_ovr + tok : NULL,
                     m_ovr ? m_ovr + tok : NULL, full, out ? out + tok * dv : NULL,
                     b_out ? b_out + tok : NULL, merge_out ? merge_out + tok : NULL,
                     score_out ? score_out + tok : NULL, m_out ? m_out + tok : NULL,
                     margin_b ? margin_b + tok : NULL, margin_m ? margin_m + tok : NULL,
                     mag_out ? mag_out + tok : NULL, u_out ? u_out + tok * dv : NULL,
                     cache_m + h, cache_n + h * C,
                     cache_ibar + h * C, cache_S + h * C * D);
    if (r != ORACLE_OK) {
#pragma omp critical
      rc = r;
    }
  }
  return rc;
}
