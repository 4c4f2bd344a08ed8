/*
 * Oracle for the Gated DeltaNet (GDN) state recurrence -- TEST INFRASTRUCTURE.
 *
 * Only tests, the smoke check and the CPU-baseline leg of the benchmark may
 * load this library.  The product path (the HIP library) never does.
 *
 * What it computes (fp64 throughout, token by token, no chunking):
 *
 *   Paper, Section 2, Eq. (1):  S_i = T_i S_{i-1} + beta_i v_i k_i^T,
 *                               T_i = alpha_i (I - beta_i k_i k_i^T),
 *   read as S in R^{d_v x d_k} with the transition applied on the key side,
 *       S_i = S_{i-1} alpha_i (I - beta_i k_i k_i^T) + beta_i v_i k_i^T,
 *   and stored transposed, M = S^T in R^{d_k x d_v} (row-major, d_v fastest):
 *       M_i = alpha_i M_{i-1} + k_i (beta_i (v_i - alpha_i M_{i-1}^T k_i))^T.
 *   alpha_i = exp(g_i) with g_i = log alpha_i passed in per token and value head.
 *
 *   Paper, Section 3, Eq. (2) (Independent Tail-Replay): the replay starts from
 *   a zero state at the beginning of the tail and applies Eq. (1) to every tail
 *   token; the state after the last tail token is the rebuilt state.  Here that
 *   is a call with state_in == NULL over the tail tokens.
 *
 *   Outputs (not printed in the paper; the usual GDN read-out): after the update
 *   of token t, o_t = scale * S_t q_t = scale * M_t^T q_t.
 *
 *   Grouped heads: value head h reads query/key head h / (Hv / Hk).
 *
 * Parallelism: OpenMP over independent (sequence, value head) units only; each
 * unit is the plain sequential loop above.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One (sequence, value head) unit.  M is caller-provided scratch [dk*dv],
 * p and w are scratch [dv]. */
static void gdn_oracle_unit(int64_t t0, int64_t t1, int32_t hk, int32_t hv,
                            int32_t dk, int32_t dv, int32_t h, int32_t kh,
                            const double* q, const double* k, const double* v,
                            const double* g, const double* beta,
                            const double* m_in, double scale, double* o,
                            double* m_out, double* M, double* p, double* w) {
  const int64_t dkv = (int64_t)dk * dv;
  if (m_in)
    memcpy(M, m_in, sizeof(double) * dkv);
  else
    memset(M, 0, sizeof(double) * dkv);

  for (int64_t t = t0; t < t1; ++t) {
    const double a = exp(g[t * hv + h]);
    const double b = beta[t * hv + h];
    const double* kt = k + (t * hk + kh) * dk;
    const double* vt = v + (t * hv + h) * dv;

    /* p = M^T k  (= S k, the value the state currently recalls for key k) */
    for (int32_t c = 0; c < dv; ++c) p[c] = 0.0;
    for (int32_t d = 0; d < dk; ++d) {
      const double kd = kt[d];
      const double* row = M + (int64_t)d * dv;
      for (int32_t c = 0; c < dv; ++c) p[c] += kd * row[c];
    }
    /* w = beta (v - alpha p): the delta written along k */
    for (int32_t c = 0; c < dv; ++c) w[c] = b * (vt[c] - a * p[c]);
    /* M = alpha M + k w^T */
    for (int32_t d = 0; d < dk; ++d) {
      const double kd = kt[d];
      double* row = M + (int64_t)d * dv;
      for (int32_t c = 0; c < dv; ++c) row[c] = a * row[c] + kd * w[c];
    }
    if (o) {
      const double* qt = q + (t * hk + kh) * dk;
      double* ot = o + (t * hv + h) * dv;
      for (int32_t c = 0; c < dv; ++c) ot[c] = 0.0;
      for (int32_t d = 0; d < dk; ++d) {
        const double qd = qt[d];
        const double* row = M + (int64_t)d * dv;
        for (int32_t c = 0; c < dv; ++c) ot[c] += qd * row[c];
      }
      for (int32_t c = 0; c < dv; ++c) ot[c] *= scale;
    }
  }
  memcpy(m_out, M, sizeof(double) * dkv);
}

/*
 * Runs the recurrence for every (sequence, value head).
 *
 *   cu_seqlens [N+1]      token offsets of the packed sequences (host memory)
 *   q          [T,Hk,dk]  or NULL: then o must be NULL too
 *   k          [T,Hk,dk]
 *   v          [T,Hv,dv]
 *   g, beta    [T,Hv]     log-gate and write strength
 *   state_in   [N,Hv,dk,dv] or NULL for the zero state
 *   o          [T,Hv,dv]  or NULL
 *   state_out  [N,Hv,dk,dv]
 *   nthreads   OpenMP threads (<= 0: library default)
 *
 * Returns 0, or a negative code for inconsistent arguments (nothing written).
 */
int gdn_oracle_recurrence(int32_t num_seqs, int32_t hk, int32_t hv, int32_t dk,
                          int32_t dv, const int64_t* cu_seqlens,
                          const double* q, const double* k, const double* v,
                          const double* g, const double* beta,
                          const double* state_in, double scale, double* o,
                          double* state_out, int32_t nthreads) {
  if (num_seqs < 0 || hk <= 0 || hv <= 0 || dk <= 0 || dv <= 0) return -1;
  if (hv % hk != 0) return -2;
  if (!cu_seqlens || !k || !v || !g || !beta || !state_out) return -3;
  if ((o != NULL) != (q != NULL)) return -4;
  if (cu_seqlens[0] != 0) return -5;
  for (int32_t n = 0; n < num_seqs; ++n)
    if (cu_seqlens[n + 1] < cu_seqlens[n]) return -5;

  const int32_t grp = hv / hk;
  const int64_t units = (int64_t)num_seqs * hv;
  const int64_t dkv = (int64_t)dk * dv;
  int failed = 0;

#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads) reduction(| : failed)
#endif
  {
    double* M = (double*)malloc(sizeof(double) * (dkv + 2 * (int64_t)dv));
    if (!M) {
      failed = 1;
    } else {
      double* p = M + dkv;
      double* w = p + dv;
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t u = 0; u < units; ++u) {
        const int32_t n = (int32_t)(u / hv);
        const int32_t h = (int32_t)(u % hv);
        gdn_oracle_unit(cu_seqlens[n], cu_seqlens[n + 1], hk, hv, dk, dv, h,
                        h / grp, q, k, v, g, beta,
                        state_in ? state_in + u * dkv : NULL, scale, o,
                        state_out + u * dkv, M, p, w);
      }
      free(M);
    }
  }
  (void)nthreads;
  return failed ? -6 : 0;
}

/* Number of OpenMP threads the library would use by default. */
int gdn_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
