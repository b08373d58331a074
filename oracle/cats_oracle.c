/*
 * CATS CPU oracle -- TEST INFRASTRUCTURE ONLY (see cats_oracle.h).
 *
 * Written from the paper's definitions, in its order and notation:
 *   Eq. 1  Gated-MLP(x) = (SiLU(x W_gate) * (x W_up)) W_down
 *   Eq. 2  SiLU(z) = z * sigmoid(z) = z / (1 + e^{-z})
 *   Eq. 3  t = min{t' : F(t') >= k}, F the empirical CDF of |activations|
 *   Eq. 4/5 CATS_t keeps an activation when |.| >= t, else zeroes it
 *   Section 4.3, "MLP using CATS": v = SiLU(x W_gate); Mask = |v| >= t;
 *          x1 = (x W_up[Mask]) * v[Mask]; y = x1 W_down[Mask]
 * Nothing here is blocked, fused or reordered beyond those definitions:
 * every sum runs over its index in ascending order starting from +0.
 *
 * Readings where the paper is silent or inconsistent:
 *   - The comparison keeps ties (|v| >= t), as Eq. 4, Eq. 5 and all three
 *     kernel algorithms write it; the appendix restatement with a strict
 *     ">" is taken as a typo.  It is evaluated as !(|v| < t), so a NaN
 *     activation is kept and t = 0 keeps everything.
 *   - The cutoff is one scalar per MLP block, pooled over every calibration
 *     vector and every neuron; the quantile is the order statistic of rank
 *     ceil(k n) with no interpolation, and k = 0 gives t = 0.
 */
#include "cats_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifdef ORACLE_F64
typedef double real;
#define R_EXP exp
#define R_SQRT sqrt
#define R_FABS fabs
static const char* k_precision = "f64";
#else
typedef float real;
#define R_EXP expf
#define R_SQRT sqrtf
#define R_FABS fabsf
static const char* k_precision = "f32";
#endif

const char* oracle_precision(void) { return k_precision; }

/* Threads: an OpenMP build (-fopenmp) splits independent outputs over
 * threads -- the neurons of x W_gate and x W_up, the columns of the
 * down-projection, the calibration vectors -- and never a sum, so every
 * value is computed by the same operations in the same order as in the
 * sequential build, bit for bit. */
int oracle_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

/* This thread's share [*lo, *hi) of n independent outputs (all of them in
 * a sequential build or outside a parallel region). */
static void thread_share(int32_t n, int32_t* lo, int32_t* hi) {
#ifdef _OPENMP
  const int64_t nt = omp_get_num_threads(), t = omp_get_thread_num();
  *lo = (int32_t)(n * t / nt);
  *hi = (int32_t)(n * (t + 1) / nt);
#else
  *lo = 0;
  *hi = n;
#endif
}

/* Eq. 2. */
static real silu(real z) { return z / ((real)1 + R_EXP(-z)); }

double oracle_silu(double z) { return (double)silu((real)z); }

/* Eq. 4: CATS_t keeps z when |z| >= t. */
static int cats_keeps(real v, real t) { return !(R_FABS(v) < t); }

int oracle_cats_mlp(const float* x, int32_t B, int32_t d, int32_t m,
                    const float* w_gate, const float* w_up, const float* w_down,
                    double t_in, int32_t dense, const float* residual,
                    double* y, int32_t* active_idx, int32_t* active_cnt,
                    double* v_all, double* h_act) {
  if (!x || !w_gate || !w_up || !w_down || !y || B <= 0 || d <= 0 || m <= 0) return -1;
  if (t_in != t_in || t_in < 0) return -1;
  const real t = (real)t_in;
  real* g = (real*)malloc(sizeof(real) * (size_t)m);
  real* u = (real*)malloc(sizeof(real) * (size_t)m);
  real* s = (real*)malloc(sizeof(real) * (size_t)d);
  int32_t* act = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);
  real* hv = (real*)malloc(sizeof(real) * (size_t)m);
  if (!g || !u || !s || !act || !hv) { free(g); free(u); free(s); free(act); free(hv); return -1; }

  for (int32_t b = 0; b < B; ++b) {
    const float* xb = x + (size_t)b * d;
    /* g = x W_gate and u = x W_up.  The loops run i outermost so that the
     * weights are read row by row; each g_j and u_j still accumulates its
     * d terms in ascending i, starting from +0. */
#ifdef _OPENMP
#pragma omp parallel
#endif
    {
      int32_t j0, j1;
      thread_share(m, &j0, &j1);
      for (int32_t j = j0; j < j1; ++j) { g[j] = 0; u[j] = 0; }
      for (int32_t i = 0; i < d; ++i) {
        const real xi = (real)xb[i];
        const float* wg_row = w_gate + (size_t)i * m;
        const float* wu_row = w_up + (size_t)i * m;
        for (int32_t j = j0; j < j1; ++j) {
          g[j] += xi * (real)wg_row[j];
          u[j] += xi * (real)wu_row[j];
        }
      }
    }
    /* v = SiLU(g); Mask; x1 = u[Mask] * v[Mask], listed in ascending j. */
    int32_t cnt = 0;
    for (int32_t j = 0; j < m; ++j) {
      const real v = silu(g[j]);
      if (v_all) v_all[(size_t)b * m + j] = (double)v;
      if (!(dense || cats_keeps(v, t))) continue;
      const real h = v * u[j];
      if (active_idx) active_idx[(size_t)b * m + cnt] = j;
      if (h_act) h_act[(size_t)b * m + cnt] = (double)h;
      act[cnt] = j;
      hv[cnt] = h;
      ++cnt;
    }
    if (active_cnt) active_cnt[b] = cnt;
    /* s = x1 W_down[Mask]: s_k accumulates the active j in ascending
     * order, from +0. */
#ifdef _OPENMP
#pragma omp parallel
#endif
    {
      int32_t k0, k1;
      thread_share(d, &k0, &k1);
      for (int32_t k = k0; k < k1; ++k) s[k] = 0;
      for (int32_t q = 0; q < cnt; ++q) {
        const int32_t j = act[q];
        const real h = hv[q];
        const float* wd_row = w_down + (size_t)j * d;
        for (int32_t k = k0; k < k1; ++k) s[k] += h * (real)wd_row[k];
      }
    }
    for (int32_t k = 0; k < d; ++k) {
      real out = s[k];
      if (residual) out = (real)residual[(size_t)b * d + k] + out;
      y[(size_t)b * d + k] = (double)out;
    }
  }
  free(g); free(u); free(s); free(act); free(hv);
  return 0;
}

int oracle_rmsnorm(const float* x, int32_t B, int32_t d, double eps, double* out) {
  if (!x || !out || B <= 0 || d <= 0 || !(eps >= 0)) return -1;
  for (int32_t b = 0; b < B; ++b) {
    const float* xb = x + (size_t)b * d;
    real ss = 0;
    for (int32_t i = 0; i < d; ++i) ss += (real)xb[i] * (real)xb[i];
    const real inv = (real)1 / R_SQRT(ss / (real)d + (real)eps);
    for (int32_t i = 0; i < d; ++i) out[(size_t)b * d + i] = (double)((real)xb[i] * inv);
  }
  return 0;
}

int oracle_topk_thresholds(const float* x, int32_t B, int32_t d, int32_t m, const float* w_gate,
                           double k, double* t_out) {
  if (!x || !w_gate || !t_out || B <= 0 || d <= 0 || m <= 0 || !(k >= 0.0 && k <= 1.0)) return -1;
  const int64_t r = oracle_cutoff_rank(m, k);
  double* a = (double*)malloc(sizeof(double) * (size_t)m);
  if (!a) return -1;
  for (int32_t b = 0; b < B; ++b) {
    if (r == 0) {
      t_out[b] = 0.0;
      continue;
    }
    if (oracle_calib_acts(x + (size_t)b * d, 1, d, m, w_gate, a) != 0) {
      free(a);
      return -1;
    }
    if (oracle_threshold(a, m, k, &t_out[b]) != 0) {
      free(a);
      return -1;
    }
  }
  free(a);
  return 0;
}

int oracle_sparse_input_gemv(const float* x, int32_t B, int32_t d, int32_t n, const float* w,
                             double t_in, const float* residual, double* y, int32_t* active_idx,
                             int32_t* active_cnt) {
  if (!x || !w || !y || B <= 0 || d <= 0 || n <= 0) return -1;
  if (t_in != t_in || t_in < 0) return -1;
  const real t = (real)t_in;
  real* s = (real*)malloc(sizeof(real) * (size_t)n);
  if (!s) return -1;
  for (int32_t b = 0; b < B; ++b) {
    const float* xb = x + (size_t)b * d;
    for (int32_t k = 0; k < n; ++k) s[k] = 0;
    int32_t cnt = 0;
    for (int32_t i = 0; i < d; ++i) {
      const real xc = (real)xb[i];
      if (!cats_keeps(xc, t)) continue;
      if (active_idx) active_idx[(size_t)b * d + cnt] = i;
      ++cnt;
      const float* w_row = w + (size_t)i * n;
      for (int32_t k = 0; k < n; ++k) s[k] += xc * (real)w_row[k];
    }
    if (active_cnt) active_cnt[b] = cnt;
    for (int32_t k = 0; k < n; ++k) {
      real out = s[k];
      if (residual) out = (real)residual[(size_t)b * n + k] + out;
      y[(size_t)b * n + k] = (double)out;
    }
  }
  free(s);
  return 0;
}

int oracle_stack(const float* x0, int32_t B, int32_t d, int32_t m, int32_t L,
                 const float* const* w_gate, const float* const* w_up,
                 const float* const* w_down, const double* t, int32_t dense, double eps,
                 float* x_all, int32_t* active_cnt) {
  if (!x0 || !w_gate || !w_up || !w_down || !x_all || B <= 0 || d <= 0 || m <= 0 || L < 0)
    return -1;
  if (!dense && !t) return -1;
  const size_t n = (size_t)B * d;
  double* tmp = (double*)malloc(sizeof(double) * n);
  float* xn = (float*)malloc(sizeof(float) * n);
  double* y = (double*)malloc(sizeof(double) * n);
  int32_t* cnt = (int32_t*)malloc(sizeof(int32_t) * (size_t)B);
  int rc = (tmp && xn && y && cnt) ? 0 : -1;
  if (rc == 0) memcpy(x_all, x0, sizeof(float) * n);
  for (int32_t l = 0; l < L && rc == 0; ++l) {
    const float* xl = x_all + (size_t)l * n;
    float* xnext = x_all + (size_t)(l + 1) * n;
    rc = oracle_rmsnorm(xl, B, d, eps, tmp);
    if (rc != 0) break;
    for (size_t i = 0; i < n; ++i) xn[i] = (float)tmp[i];
    rc = oracle_cats_mlp(xn, B, d, m, w_gate[l], w_up[l], w_down[l], dense ? 0.0 : t[l], dense, xl,
                         y, NULL, cnt, NULL, NULL);
    if (rc != 0) break;
    for (size_t i = 0; i < n; ++i) xnext[i] = (float)y[i];
    if (active_cnt) memcpy(active_cnt + (size_t)l * B, cnt, sizeof(int32_t) * (size_t)B);
  }
  free(tmp);
  free(xn);
  free(y);
  free(cnt);
  return rc;
}

/* |SiLU(x_n . Wg[:,j])|, the activation whose CDF defines the cutoff. */
static real calib_act(const float* xn, int32_t d, int32_t m, const float* w_gate, int32_t j) {
  real g = 0;
  for (int32_t i = 0; i < d; ++i) g += (real)xn[i] * (real)w_gate[(size_t)i * m + j];
  return R_FABS(silu(g));
}

int oracle_calib_acts(const float* X, int32_t N, int32_t d, int32_t m,
                      const float* w_gate, double* acts) {
  if (!X || !w_gate || !acts || N <= 0 || d <= 0 || m <= 0) return -1;
  int failed = 0;
#ifdef _OPENMP
#pragma omp parallel
#endif
  {
    real* g = (real*)malloc(sizeof(real) * (size_t)m);
    int32_t n0, n1;
    thread_share(N, &n0, &n1);
    if (!g) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      failed = 1;
      n1 = n0;
    }
    for (int32_t n = n0; n < n1; ++n) {
      const float* xn = X + (size_t)n * d;
      /* Same ascending-i accumulation as calib_act, with i outermost. */
      for (int32_t j = 0; j < m; ++j) g[j] = 0;
      for (int32_t i = 0; i < d; ++i) {
        const real xi = (real)xn[i];
        const float* row = w_gate + (size_t)i * m;
        for (int32_t j = 0; j < m; ++j) g[j] += xi * (real)row[j];
      }
      for (int32_t j = 0; j < m; ++j) acts[(size_t)n * m + j] = (double)R_FABS(silu(g[j]));
    }
    free(g);
  }
  return failed ? -1 : 0;
}

int oracle_calib_acts_at(const float* X, int32_t N, int32_t d, int32_t m,
                         const float* w_gate, const int64_t* pairs,
                         int64_t npairs, double* out) {
  if (!X || !w_gate || !pairs || !out || N <= 0 || d <= 0 || m <= 0 || npairs < 0) return -1;
  for (int64_t q = 0; q < npairs; ++q) {
    const int64_t n = pairs[2 * q], j = pairs[2 * q + 1];
    if (n < 0 || n >= N || j < 0 || j >= m) return -1;
    out[q] = (double)calib_act(X + (size_t)n * d, d, m, w_gate, (int32_t)j);
  }
  return 0;
}

int64_t oracle_cutoff_rank(int64_t n, double k) {
  if (n <= 0 || !(k >= 0.0 && k <= 1.0)) return -1;
  if (k == 0.0) return 0;
  /* F(t') >= k  <=>  #{|a| <= t'} >= k n; the smallest such t' is the
   * order statistic of rank ceil(k n).  The 1e-6 guard keeps an exact
   * product such as 0.7 * 1000 from rounding up past its integer. */
  double r = ceil(k * (double)n - 1e-6);
  if (r < 1) r = 1;
  if (r > (double)n) r = (double)n;
  return (int64_t)r;
}

/* Ascending order on |a|; NaN sorts after every number. */
static int cmp_abs(const void* pa, const void* pb) {
  const double a = fabs(*(const double*)pa), b = fabs(*(const double*)pb);
  const int an = a != a, bn = b != b;
  if (an || bn) return an - bn;
  return (a > b) - (a < b);
}

int oracle_threshold(const double* a, int64_t n, double k, double* t) {
  if (!a || !t || n <= 0) return -1;
  const int64_t r = oracle_cutoff_rank(n, k);
  if (r < 0) return -1;
  if (r == 0) { *t = 0.0; return 0; }
  double* c = (double*)malloc(sizeof(double) * (size_t)n);
  if (!c) return -1;
  memcpy(c, a, sizeof(double) * (size_t)n);
  qsort(c, (size_t)n, sizeof(double), cmp_abs);
  *t = fabs(c[r - 1]);
  free(c);
  return 0;
}
