/*
 * CATS CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, sequential CPU implementation of what the CATS gated-MLP
 * computes (Lee et al., "CATS: Contextually-Aware Thresholding for Sparsity
 * in Large Language Models", COLM 2024).  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this library; the
 * product path (libcats) never links or calls it, and the two share no
 * code, header or helper.
 *
 * Precision: the paper runs all experiments in FP32 (Section 5, setup), so
 * the default build accumulates in float with a strictly ascending index
 * order and no fused multiply-add (-O2 -ffp-contract=off, no fast-math).
 * Building with -DORACLE_F64 gives the same code in double, which bounds
 * the float build's own rounding.
 *
 * Layouts follow the paper's notation (Section 3, Eq. 1):
 *   x       [B x d]   row-major
 *   w_gate  [d x m]   row-major (math layout, element (i,j) at i*m + j)
 *   w_up    [d x m]   row-major
 *   w_down  [m x d]   row-major (element (j,k) at j*d + k)
 * All pointers are host pointers owned by the caller.
 */
#ifndef CATS_ORACLE_H
#define CATS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Name of the accumulation type this copy was compiled with: "f32" or "f64". */
const char* oracle_precision(void);

/* Threads of an OpenMP build (-fopenmp): sets the count when n > 0 and
 * returns the count in use (1 in a sequential build).  Threads split
 * independent outputs only, so results are bit-identical to the
 * sequential build. */
int oracle_threads(int n);

/* SiLU(z) = z / (1 + exp(-z)) (Eq. 2), evaluated in the build's precision. */
double oracle_silu(double z);

/* The gated MLP with the CATS activation (Eq. 1 with Eq. 5, and the
 * "MLP using CATS" algorithm of Section 4.3).  For every row b:
 *   g_j = sum_i x_bi Wg[i,j],  u_j = sum_i x_bi Wu[i,j]   (ascending i)
 *   v_j = SiLU(g_j)
 *   neuron j is active when |v_j| >= t   (written !(|v_j| < t); Eq. 4)
 *   s_k = sum over active j, ascending, of (v_j u_j) Wd[j,k]   (from +0)
 *   y_bk = residual_bk + s_k     (residual may be NULL: y = s)
 * dense != 0 keeps every neuron (plain Eq. 1).  t = 0 keeps every neuron as
 * well, so it reproduces dense bit for bit.
 * Optional outputs (NULL to skip), per row b, in ascending neuron order:
 *   active_idx[b*m + q], active_cnt[b], v_all[b*m + j] (every j),
 *   h_act[b*m + q] = v_j u_j of the q-th active neuron.
 * Returns 0, or -1 on a bad argument. */
int oracle_cats_mlp(const float* x, int32_t B, int32_t d, int32_t m,
                    const float* w_gate, const float* w_up, const float* w_down,
                    double t, int32_t dense, const float* residual,
                    double* y, int32_t* active_idx, int32_t* active_cnt,
                    double* v_all, double* h_act);

/* RMSNorm with unit gain: out_bi = x_bi / sqrt(mean_i(x_bi^2) + eps),
 * the sum of squares taken in ascending i. */
int oracle_rmsnorm(const float* x, int32_t B, int32_t d, double eps, double* out);

/* Per-token cutoffs for a top-k variant of CATS (the paper's future work:
 * a minimum sparsity per token instead of one calibrated t): for every row
 * b, v_j = SiLU(x_b . Wg[:, j]) over the m neurons and
 *   t_out[b] = the r-th smallest |v_j| (1-indexed), r = oracle_cutoff_rank(m, k)
 * i.e. Eq. 3 applied to the token's own m activations.  CATS with t_out[b]
 * on row b then keeps the neurons with |v_j| >= t_out[b]: at least m - r + 1
 * of them (ties kept).  k = 0 gives 0.  Returns 0, or -1 on a bad argument. */
int oracle_topk_thresholds(const float* x, int32_t B, int32_t d, int32_t m, const float* w_gate,
                           double k, double* t_out);

/* CATS on the input of a linear layer (Appendix B wraps the attention
 * block's input x in CATS_t): y_b = residual_b + CATS_t(x_b) W with
 * CATS_t(z) = z where |z| >= t, else 0 (Eq. 4).  W is [d x n] row-major, row
 * i holding input channel i's n output weights.  For every row b the kept
 * channels are taken in ascending i and s_k = sum_i x_bi W[i, k] accumulates
 * from +0; y_bk = residual_bk + s_k (residual may be NULL).  Optional:
 * active_idx[b*d + q] (ascending kept channels), active_cnt[b].  t = 0 keeps
 * every channel (a plain product).  Returns 0, or -1 on a bad argument. */
int oracle_sparse_input_gemv(const float* x, int32_t B, int32_t d, int32_t n, const float* w,
                             double t, const float* residual, double* y, int32_t* active_idx,
                             int32_t* active_cnt);

/* Residual stack of L gated-MLP blocks, the MLP half of a decoder's layers
 * (norms and residuals sit outside the paper's formulas, Appendix B).  For
 * l = 0 .. L-1 and every row b:
 *   xn      = RMSNorm(x_l)          unit gain, epsilon eps
 *   x_{l+1} = x_l + MLP_l(xn)       MLP_l: oracle_cats_mlp at t[l], or
 *                                   dense for every layer when dense != 0
 * The residual stream is a float vector between layers: xn and x_{l+1} are
 * stored as float (exact in the f32 build, rounded in the f64 build).
 * w_gate[l], w_up[l], w_down[l] point at layer l's math-layout weights,
 * every layer d x m.  x_all [(L+1) x B x d] receives x_0 .. x_L;
 * active_cnt [L x B] (NULL to skip) the kept neurons of every layer and
 * row.  Returns 0, or -1 on a bad argument. */
int oracle_stack(const float* x0, int32_t B, int32_t d, int32_t m, int32_t L,
                 const float* const* w_gate, const float* const* w_up,
                 const float* const* w_down, const double* t, int32_t dense, double eps,
                 float* x_all, int32_t* active_cnt);

/* Calibration activations (Section 4.1): a[n*m + j] = |SiLU(x_n . Wg[:,j])|
 * for N calibration vectors. */
int oracle_calib_acts(const float* X, int32_t N, int32_t d, int32_t m,
                      const float* w_gate, double* acts);

/* The same activations for an explicit list of (n, j) pairs
 * (pairs[2q] = n, pairs[2q+1] = j), for sampled checks at full size. */
int oracle_calib_acts_at(const float* X, int32_t N, int32_t d, int32_t m,
                         const float* w_gate, const int64_t* pairs,
                         int64_t npairs, double* out);

/* Rank of the cutoff order statistic for sparsity k over n values
 * (Eq. 3 on the empirical CDF): r = ceil(k*n - 1e-6) clamped to [1, n].
 * Returns 0 when k == 0 (the cutoff is then t = 0).  -1 on bad input. */
int64_t oracle_cutoff_rank(int64_t n, double k);

/* Cutoff threshold t = min{t' : F(t') >= k} (Eq. 3), F the empirical CDF of
 * |a| over the n given values: the r-th smallest |a| (1-indexed), found by
 * sorting a copy.  k == 0 gives 0.  Returns 0 and writes *t, or -1. */
int oracle_threshold(const double* a, int64_t n, double k, double* t);

#ifdef __cplusplus
}
#endif
#endif
