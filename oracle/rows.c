/*
 * CPU oracle, per-row part: reverse KL between the student and teacher
 * next-token distributions over the full vocabulary, and its derivative with
 * respect to the student logits, in float64.
 *
 * TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
 * cpu_baseline leg may load this library.  It shares no code with the HIP
 * path.
 *
 * Definitions followed (TurnOPD, arXiv 2607.05804):
 *   - Sec. 3 (Preliminaries), Eq. (opd-rkl): the per-token loss is the reverse
 *     KL D_KL(pi_theta(.|s_i) || pi_T(.|s_i)) = sum_v p_s(v) (log p_s(v) - log p_t(v)),
 *     student first.
 *   - App. D (Complete TurnOPD Hyperparameters), full-configuration table:
 *     training temperature 1.0, so the logits are used unscaled:
 *     log p(v) = z(v) - log sum_u exp z(u).
 *   - The teacher is frozen (Sec. 3), so only the student logits receive a
 *     gradient.  With p = p_s and d_v = log p_s(v) - log p_t(v):
 *       dKL/dz_s(j) = p_j d_j - p_j sum_v p_v d_v = p_j (d_j - KL),
 *     since d log p_s(v) / d z_s(j) = [v == j] - p_j.
 *
 * Computation (plain two-pass definition, no one-pass recurrences):
 *   lse = m + log sum_v exp(z_v - m), m = max_v z_v   (student and teacher)
 *   ls_v = zs_v - lse_s,  lt_v = zt_v - lse_t,  p_v = exp(ls_v)
 *   KL   = sum_v p_v (ls_v - lt_v)                   (summed in index order)
 *   g_v  = p_v (ls_v - lt_v - KL)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* dtype codes: 0 = bfloat16 (stored as its 16-bit pattern), 1 = float32,
 * 2 = float64 (used by the finite-difference checks). */
static double widen(const void* base, int dtype, int64_t idx) {
  if (dtype == 0) {
    const uint32_t u = (uint32_t)((const uint16_t*)base)[idx] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f; /* bf16 -> fp32 -> fp64 is exact */
  }
  if (dtype == 1) return (double)((const float*)base)[idx];
  return ((const double*)base)[idx];
}

/* log sum_v exp(z_v), evaluated as m + log sum_v exp(z_v - m). */
static double log_sum_exp(const double* z, int64_t V) {
  double m = z[0];
  for (int64_t v = 1; v < V; ++v)
    if (z[v] > m) m = z[v];
  double s = 0.0;
  for (int64_t v = 0; v < V; ++v) s += exp(z[v] - m);
  return m + log(s);
}

/*
 * For each of n_rows rows: zs + r*ld_s and zt + r*ld_t hold V logits.
 *   kl_out[r]           <- KL(p_s || p_t)
 *   g_out + r*ld_g      <- dKL/dz_s (V values), when g_out != NULL
 *   lse_out[2r], [2r+1] <- lse_s, lse_t (the log-partition functions of the
 *                          two rows), when lse_out != NULL
 * Rows are independent; they are spread over n_threads OpenMP threads
 * (<= 0: the OpenMP default).  Returns 0, or -1 on a bad argument / OOM.
 */
int oracle_rows(const void* zs, int64_t ld_s, const void* zt, int64_t ld_t, int dtype,
                int64_t n_rows, int64_t V, double* kl_out, double* g_out, int64_t ld_g,
                double* lse_out, int n_threads) {
  if (!zs || !zt || !kl_out || V < 1 || n_rows < 0 || ld_s < V || ld_t < V) return -1;
  if (dtype < 0 || dtype > 2) return -1;
  if (g_out && ld_g < V) return -1;
  int failed = 0;
#ifdef _OPENMP
  const int nt = n_threads > 0 ? n_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt) reduction(| : failed)
#endif
  for (int64_t r = 0; r < n_rows; ++r) {
    double* ls = (double*)malloc((size_t)V * sizeof(double));
    double* lt = (double*)malloc((size_t)V * sizeof(double));
    if (!ls || !lt) {
      free(ls);
      free(lt);
      failed = 1;
      continue;
    }
    for (int64_t v = 0; v < V; ++v) {
      ls[v] = widen(zs, dtype, r * ld_s + v);
      lt[v] = widen(zt, dtype, r * ld_t + v);
    }
    const double lse_s = log_sum_exp(ls, V);
    const double lse_t = log_sum_exp(lt, V);
    if (lse_out) {
      lse_out[2 * r] = lse_s;
      lse_out[2 * r + 1] = lse_t;
    }
    for (int64_t v = 0; v < V; ++v) {
      ls[v] -= lse_s; /* log p_s(v) */
      lt[v] -= lse_t; /* log p_t(v) */
    }
    double kl = 0.0;
    for (int64_t v = 0; v < V; ++v) kl += exp(ls[v]) * (ls[v] - lt[v]);
    kl_out[r] = kl;
    if (g_out) {
      double* g = g_out + r * ld_g;
      for (int64_t v = 0; v < V; ++v) g[v] = exp(ls[v]) * (ls[v] - lt[v] - kl);
    }
    free(ls);
    free(lt);
  }
  return failed ? -1 : 0;
}

/* Number of OpenMP threads a default-threaded call would use. */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
