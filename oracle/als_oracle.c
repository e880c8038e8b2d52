/*
 * fp64 CPU oracle of the ALS half-sweep -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
 * load this library. It shares no code with the HIP library: it has its own
 * transpose, its own normal equations, its own Cholesky and its own residual.
 *
 * What it computes (paper, Sec. 2.2 "ALS and BPTF"): the rating matrix A
 * (M x N, observed entries only) is approximated by U V with U (M x D) and
 * V (D x N, stored here N x D). With one side fixed, every row s of the other
 * side is the exact minimiser of
 *     sum_{j in Omega_s} (r_sj - f_j . x)^2 + lambda * n_s * ||x||^2,
 * i.e. x_s = (sum_j f_j f_j^T + lambda n_s I)^{-1} sum_j r_sj f_j, where f_j
 * are the fixed-side rows of the ratings of s and n_s = |Omega_s|. The
 * per-update inversion of Sec. 4.1 is done here as a Cholesky factorisation
 * and two triangular solves. A prediction is the dot product of the user and
 * item vectors (Sec. 2.2); RMSE (Sec. 4.1) is sqrt(sum of squared residuals /
 * number of ratings) over the stored ratings.
 *
 * Weighted ALS (the paper's wALS, listed with ALS in Sec. 2 and Sec. 4, whose
 * weighting the paper does not define): with a non-negative weight c_sj on every
 * stored rating, the row minimises sum_j c_sj (r_sj - f_j . x)^2 + lambda n_s ||x||^2,
 * so x_s = (sum_j c_sj f_j f_j^T + lambda n_s I)^{-1} sum_j c_sj r_sj f_j; the
 * regulariser keeps the count n_s, so unit weights give plain ALS. Every function
 * that takes a weight array wt treats NULL as the unweighted method.
 *
 * Held-out prediction (Sec. 2.2 prediction; Sec. 4.1 measures the RMSE on
 * validation ratings that training did not see): for a list of (user, item)
 * pairs, r_hat = u_u . v_i, and the validation RMSE is
 * sqrt(sum over the pairs of (r - r_hat)^2 / number of pairs).
 *
 * Everything is double precision, sequential within a row, rows in parallel
 * (OpenMP). Reductions over rows are done in row order from per-row values,
 * so every result is independent of the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

static void set_threads(int nthreads) {
  if (nthreads > 0) omp_set_num_threads(nthreads);
}

/* Compressed rows -> compressed columns by counting; rows stay ascending
 * within each column. out_ptr has n_cols + 1 entries. Returns 0 or -1. */
int orc_transpose(int64_t n_rows, int64_t n_cols, const int64_t *ptr, const int32_t *idx,
                  const double *val, int64_t *out_ptr, int32_t *out_idx, double *out_val) {
  for (int64_t c = 0; c <= n_cols; ++c) out_ptr[c] = 0;
  for (int64_t p = 0; p < ptr[n_rows]; ++p) {
    if (idx[p] < 0 || idx[p] >= n_cols) return -1;
    out_ptr[idx[p] + 1] += 1;
  }
  for (int64_t c = 0; c < n_cols; ++c) out_ptr[c + 1] += out_ptr[c];
  int64_t *next = (int64_t *)malloc(sizeof(int64_t) * (n_cols > 0 ? n_cols : 1));
  if (!next) return -1;
  for (int64_t c = 0; c < n_cols; ++c) next[c] = out_ptr[c];
  for (int64_t r = 0; r < n_rows; ++r) {
    for (int64_t p = ptr[r]; p < ptr[r + 1]; ++p) {
      int64_t q = next[idx[p]];
      next[idx[p]] = q + 1;
      out_idx[q] = (int32_t)r;
      out_val[q] = val[p];
    }
  }
  free(next);
  return 0;
}

/* Normal equations of one row: A = sum_k c_k f_k f_k^T + lambda * n * I (full
 * D x D, row-major) and b = sum_k c_k r_k f_k, accumulated in the order of the
 * row's ratings; c_k = wt[k], or 1 when wt is NULL. */
void orc_normal_equations(int32_t D, int64_t n, const int32_t *idx, const double *val,
                          const double *wt, const double *F, double lambda, double *A,
                          double *b) {
  for (int32_t a = 0; a < D * D; ++a) A[a] = 0.0;
  for (int32_t a = 0; a < D; ++a) b[a] = 0.0;
  for (int64_t k = 0; k < n; ++k) {
    const double *f = F + (int64_t)idx[k] * D;
    double r = val[k];
    for (int32_t a = 0; a < D; ++a) {
      const double cf = wt ? wt[k] * f[a] : f[a];
      for (int32_t e = 0; e < D; ++e) A[a * D + e] += cf * f[e];
      b[a] += r * cf;
    }
  }
  for (int32_t a = 0; a < D; ++a) A[a * D + a] += lambda * (double)n;
}

/* Solve A x = b for symmetric positive definite A (D x D, row-major; only the
 * lower triangle is read) by Cholesky A = L L^T, then L y = b and L^T x = y.
 * L is written to the lower triangle of W (D x D scratch). Returns 0, or 1
 * if a pivot is not strictly positive or not finite (x untouched). */
int orc_cholesky_solve(int32_t D, const double *A, const double *b, double *W, double *x) {
  for (int32_t i = 0; i < D; ++i) {
    for (int32_t j = 0; j <= i; ++j) {
      double s = A[i * D + j];
      for (int32_t m = 0; m < j; ++m) s -= W[i * D + m] * W[j * D + m];
      if (i == j) {
        if (!(s > 0.0) || !isfinite(s)) return 1;
        W[i * D + i] = sqrt(s);
      } else {
        W[i * D + j] = s / W[j * D + j];
      }
    }
  }
  double *y = (double *)malloc(sizeof(double) * (D > 0 ? D : 1));
  if (!y) return 1;
  for (int32_t i = 0; i < D; ++i) {
    double s = b[i];
    for (int32_t m = 0; m < i; ++m) s -= W[i * D + m] * y[m];
    y[i] = s / W[i * D + i];
  }
  for (int32_t i = D - 1; i >= 0; --i) {
    double s = y[i];
    for (int32_t m = i + 1; m < D; ++m) s -= W[m * D + i] * x[m];
    x[i] = s / W[i * D + i];
  }
  for (int32_t i = 0; i < D; ++i) {
    if (!isfinite(x[i])) { free(y); return 1; }
  }
  free(y);
  return 0;
}

/* One row's update into x (length D). Returns 0 (solved), 1 (not SPD /
 * non-finite: x untouched) or 2 (no ratings: x untouched). */
static int solve_one(int32_t D, int64_t n, const int32_t *idx, const double *val,
                     const double *wt, const double *F, double lambda, double *A, double *b,
                     double *W, double *xs, double *x) {
  if (n == 0) return 2;
  orc_normal_equations(D, n, idx, val, wt, F, lambda, A, b);
  if (orc_cholesky_solve(D, A, b, W, xs) != 0) return 1;
  for (int32_t a = 0; a < D; ++a) x[a] = xs[a];
  return 0;
}

/* Half-sweep: for every row s in [0, n_rows) with the fixed side F
 * (n_fixed x D), X[s,:] <- the regularised least-squares solution. Rows with
 * no ratings and flagged rows keep their previous X. flags[s] (nullable)
 * receives 0 solved, 1 flagged, 2 empty. Returns the number of flagged rows. */
int64_t orc_half_sweep(int64_t n_rows, const int64_t *ptr, const int32_t *idx, const double *val,
                       const double *wt, int32_t D, const double *F, double lambda, double *X,
                       int8_t *flags, int nthreads) {
  set_threads(nthreads);
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *W = (double *)malloc(sizeof(double) * D * D);
    double *b = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t s = 0; s < n_rows; ++s) {
      int st = solve_one(D, ptr[s + 1] - ptr[s], idx + ptr[s], val + ptr[s],
                         wt ? wt + ptr[s] : NULL, F, lambda, A, b, W, xs, X + s * D);
      if (flags) flags[s] = (int8_t)st;
      nflag += (st == 1);
    }
    free(A); free(W); free(b); free(xs);
  }
  return nflag;
}

/* The same update for a list of rows only (sampled checks at full size).
 * X_sel is n_sel x D; rows that are empty or flagged get NaN. */
int64_t orc_solve_rows(int64_t n_sel, const int64_t *rows, const int64_t *ptr, const int32_t *idx,
                       const double *val, const double *wt, int32_t D, const double *F,
                       double lambda, double *X_sel, int8_t *flags, int nthreads) {
  set_threads(nthreads);
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *W = (double *)malloc(sizeof(double) * D * D);
    double *b = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < n_sel; ++t) {
      int64_t s = rows[t];
      double *x = X_sel + t * D;
      for (int32_t a = 0; a < D; ++a) x[a] = NAN;
      int st = solve_one(D, ptr[s + 1] - ptr[s], idx + ptr[s], val + ptr[s],
                         wt ? wt + ptr[s] : NULL, F, lambda, A, b, W, xs, x);
      if (flags) flags[t] = (int8_t)st;
      nflag += (st == 1);
    }
    free(A); free(W); free(b); free(xs);
  }
  return nflag;
}

/* Per-row sums of squared residuals c_sj (r_sj - x_s . f_j)^2 (c = 1 when wt is
 * NULL) into row_sse (nullable), and their total summed in row order. */
double orc_sse(int64_t n_rows, const int64_t *ptr, const int32_t *idx, const double *val,
               const double *wt, int32_t D, const double *X, const double *F, double *row_sse,
               int nthreads) {
  set_threads(nthreads);
  double *per = row_sse ? row_sse : (double *)malloc(sizeof(double) * (n_rows > 0 ? n_rows : 1));
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t s = 0; s < n_rows; ++s) {
    const double *x = X + s * D;
    double acc = 0.0;
    for (int64_t p = ptr[s]; p < ptr[s + 1]; ++p) {
      const double *f = F + (int64_t)idx[p] * D;
      double pred = 0.0;
      for (int32_t a = 0; a < D; ++a) pred += x[a] * f[a];
      double e = val[p] - pred;
      acc += wt ? wt[p] * (e * e) : e * e;
    }
    per[s] = acc;
  }
  double total = 0.0;
  for (int64_t s = 0; s < n_rows; ++s) total += per[s];
  if (!row_sse) free(per);
  return total;
}

/* sum_s n_s * ||X_s||^2, in row order (the weighted regulariser of one side). */
double orc_weighted_norm(int64_t n_rows, const int64_t *ptr, int32_t D, const double *X) {
  double total = 0.0;
  for (int64_t s = 0; s < n_rows; ++s) {
    double q = 0.0;
    for (int32_t a = 0; a < D; ++a) q += X[s * D + a] * X[s * D + a];
    total += (double)(ptr[s + 1] - ptr[s]) * q;
  }
  return total;
}

/* Predictions r_hat_p = u_{users[p]} . v_{items[p]} (Sec. 2.2) of n pairs, each a
 * dot product over the D features in feature order. Indices must be in range
 * (checked by the caller). */
void orc_predict(int64_t n, const int32_t *users, const int32_t *items, int32_t D,
                 const double *U, const double *V, double *out, int nthreads) {
  set_threads(nthreads);
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < n; ++p) {
    const double *u = U + (int64_t)users[p] * D;
    const double *v = V + (int64_t)items[p] * D;
    double dot = 0.0;
    for (int32_t a = 0; a < D; ++a) dot += u[a] * v[a];
    out[p] = dot;
  }
}

/* Sum over n held-out pairs of (r_p - r_hat_p)^2 (the numerator of the validation
 * RMSE of Sec. 4.1), from per-pair predictions summed in pair order. */
double orc_pair_sse(int64_t n, const int32_t *users, const int32_t *items, const double *r,
                    int32_t D, const double *U, const double *V, int nthreads) {
  double *pred = (double *)malloc(sizeof(double) * (n > 0 ? n : 1));
  if (!pred) return NAN;
  orc_predict(n, users, items, D, U, V, pred, nthreads);
  double total = 0.0;
  for (int64_t p = 0; p < n; ++p) {
    const double e = r[p] - pred[p];
    total += e * e;
  }
  free(pred);
  return total;
}
