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
 * Bayesian factorisation (BPTF, Sec. 2.2, which pairs the least-squares update with draws
 * of the factor priors' parameters; the published BPMF/BPTF Gibbs sampler): ratings are Gaussian
 * with precision alpha around u . v, each row of a side has the prior N(mu, Lambda^{-1}),
 * and (mu, Lambda) have a Normal-Wishart hyperprior. One Gibbs step for a side draws
 *   - the hyperparameters from their Normal-Wishart posterior given the side's rows
 *     (orc_nw_posterior, orc_nw_sample: Bartlett's construction of the Wishart draw);
 *   - every row from its Gaussian conditional (orc_gibbs_rows):
 *     Lambda* = Lambda + alpha sum_j f_j f_j^T, mu* = Lambda*^{-1} (alpha sum_j r_sj f_j
 *     + Lambda mu), x = mu* + L*^{-T} z with Lambda* = L* L*^T and z standard normal.
 * The standard normal, chi-square and normal variates are inputs, so a draw is a
 * deterministic function of them.
 *
 * Tensor ALS (Sec. 2.2: the ALS model extended to the tensor case with the rating's time;
 * the data carry time bins, Sec. 1): each rating has a time bin t, the prediction is the
 * three-way product sum_d U_ud V_id T_td, and the update of one mode is the ALS update
 * whose fixed vectors are the elementwise products of the other two modes' rows
 * (orc_tensor_rows: f = F1[idx1] * F2[idx2]), with the same regulariser lambda n_s.
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
/* Row order of a half-sweep's schedule: descending degree, ties by row index, so that
 * the largest rows start first and do not form the tail. Rows are independent, so the
 * order changes no result. Returns a malloc'ed array of n_rows indices, or NULL. */
typedef struct { int64_t deg, row; } deg_row;
static int by_degree_desc(const void *pa, const void *pb) {
  const deg_row *a = (const deg_row *)pa, *b = (const deg_row *)pb;
  if (a->deg != b->deg) return a->deg > b->deg ? -1 : 1;
  return a->row < b->row ? -1 : (a->row > b->row);
}
static int64_t *degree_order(int64_t n_rows, const int64_t *ptr) {
  deg_row *key = (deg_row *)malloc(sizeof(deg_row) * (n_rows > 0 ? n_rows : 1));
  int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (n_rows > 0 ? n_rows : 1));
  if (!key || !order) { free(key); free(order); return NULL; }
  for (int64_t s = 0; s < n_rows; ++s) { key[s].deg = ptr[s + 1] - ptr[s]; key[s].row = s; }
  qsort(key, (size_t)n_rows, sizeof(deg_row), by_degree_desc);
  for (int64_t t = 0; t < n_rows; ++t) order[t] = key[t].row;
  free(key);
  return order;
}

int64_t orc_half_sweep(int64_t n_rows, const int64_t *ptr, const int32_t *idx, const double *val,
                       const double *wt, int32_t D, const double *F, double lambda, double *X,
                       int8_t *flags, int nthreads) {
  set_threads(nthreads);
  int64_t *order = degree_order(n_rows, ptr);
  if (!order) return -1;
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *W = (double *)malloc(sizeof(double) * D * D);
    double *b = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < n_rows; ++t) {
      const int64_t s = order[t];
      int st = solve_one(D, ptr[s + 1] - ptr[s], idx + ptr[s], val + ptr[s],
                         wt ? wt + ptr[s] : NULL, F, lambda, A, b, W, xs, X + s * D);
      if (flags) flags[s] = (int8_t)st;
      nflag += (st == 1);
    }
    free(A); free(W); free(b); free(xs);
  }
  free(order);
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

/* ---- Bayesian (BPMF / BPTF) Gibbs step ------------------------------------------------ */

/* Lower Cholesky factor: A = L L^T (A full D x D row-major, lower triangle read; L written
 * to the lower triangle of L, upper triangle zeroed). Returns 0, or 1 if not SPD. */
static int chol_lower(int32_t D, const double *A, double *L) {
  for (int32_t i = 0; i < D; ++i)
    for (int32_t j = 0; j < D; ++j) L[i * D + j] = 0.0;
  for (int32_t i = 0; i < D; ++i) {
    for (int32_t j = 0; j <= i; ++j) {
      double s = A[i * D + j];
      for (int32_t m = 0; m < j; ++m) s -= L[i * D + m] * L[j * D + m];
      if (i == j) {
        if (!(s > 0.0) || !isfinite(s)) return 1;
        L[i * D + i] = sqrt(s);
      } else {
        L[i * D + j] = s / L[j * D + j];
      }
    }
  }
  return 0;
}

/* y = L^{-1} b (forward substitution, L lower). */
static void solve_lower(int32_t D, const double *L, const double *b, double *y) {
  for (int32_t i = 0; i < D; ++i) {
    double s = b[i];
    for (int32_t m = 0; m < i; ++m) s -= L[i * D + m] * y[m];
    y[i] = s / L[i * D + i];
  }
}

/* x = L^{-T} y (back substitution with the transpose of the lower factor). */
static void solve_lower_t(int32_t D, const double *L, const double *y, double *x) {
  for (int32_t i = D - 1; i >= 0; --i) {
    double s = y[i];
    for (int32_t m = i + 1; m < D; ++m) s -= L[m * D + i] * x[m];
    x[i] = s / L[i * D + i];
  }
}

/* Conditional draw of every row s of the solved side given the fixed side F:
 *   Lambda* = Lambda + alpha sum_j f_j f_j^T,  h = alpha sum_j r_sj f_j + Lambda mu,
 *   Lambda* = L L^T,  X[s] = L^{-T} (L^{-1} h + z_s)  (= mu* + L^{-T} z_s),
 * with z the n_rows x D standard normal variates. A row without ratings is drawn from the
 * prior. flags[s]: 0 drawn, 1 Lambda* not numerically SPD (row left unchanged). Returns
 * the number of flagged rows. */
int64_t orc_gibbs_rows(int64_t n_rows, const int64_t *ptr, const int32_t *idx, const double *val,
                       int32_t D, const double *F, double alpha, const double *Lambda,
                       const double *mu, const double *z, double *X, int8_t *flags,
                       int nthreads) {
  set_threads(nthreads);
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *L = (double *)malloc(sizeof(double) * D * D);
    double *h = (double *)malloc(sizeof(double) * D);
    double *y = (double *)malloc(sizeof(double) * D);
    double *x = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t s = 0; s < n_rows; ++s) {
      for (int32_t a = 0; a < D * D; ++a) A[a] = 0.0;
      for (int32_t a = 0; a < D; ++a) h[a] = 0.0;
      for (int64_t k = ptr[s]; k < ptr[s + 1]; ++k) {
        const double *f = F + (int64_t)idx[k] * D;
        for (int32_t a = 0; a < D; ++a) {
          for (int32_t e = 0; e < D; ++e) A[a * D + e] += f[a] * f[e];
          h[a] += val[k] * f[a];
        }
      }
      for (int32_t a = 0; a < D; ++a) {
        double lm = 0.0;
        for (int32_t e = 0; e < D; ++e) lm += Lambda[a * D + e] * mu[e];
        h[a] = alpha * h[a] + lm;
        for (int32_t e = 0; e < D; ++e) A[a * D + e] = alpha * A[a * D + e] + Lambda[a * D + e];
      }
      int st = chol_lower(D, A, L);
      if (st == 0) {
        solve_lower(D, L, h, y);
        for (int32_t a = 0; a < D; ++a) y[a] += z[s * D + a];
        solve_lower_t(D, L, y, x);
        for (int32_t a = 0; a < D; ++a) {
          if (!isfinite(x[a])) st = 1;
        }
      }
      if (st == 0) {
        for (int32_t a = 0; a < D; ++a) X[s * D + a] = x[a];
      }
      if (flags) flags[s] = (int8_t)st;
      nflag += st;
    }
    free(A); free(L); free(h); free(y); free(x);
  }
  return nflag;
}

/* Normal-Wishart posterior of (mu, Lambda) given the n rows of X (n x D) and the prior
 * (mu0, beta0, W0^{-1}, nu0), with xbar = mean of the rows and S = sum_s (x_s - xbar)
 * (x_s - xbar)^T:
 *   beta* = beta0 + n,  nu* = nu0 + n,  mu0* = (beta0 mu0 + n xbar) / (beta0 + n),
 *   W*^{-1} = W0^{-1} + S + beta0 n / (beta0 + n) (mu0 - xbar)(mu0 - xbar)^T.
 * Outputs mu_s[D], Winv_s[D x D], *beta_s, *nu_s. */
void orc_nw_posterior(int64_t n, int32_t D, const double *X, const double *mu0, double beta0,
                      const double *W0inv, double nu0, double *mu_s, double *Winv_s,
                      double *beta_s, double *nu_s) {
  double *xbar = (double *)malloc(sizeof(double) * (D > 0 ? D : 1));
  for (int32_t a = 0; a < D; ++a) {
    double t = 0.0;
    for (int64_t s = 0; s < n; ++s) t += X[s * D + a];
    xbar[a] = n > 0 ? t / (double)n : 0.0;
  }
  const double nn = (double)n;
  const double shrink = (beta0 + nn) > 0.0 ? beta0 * nn / (beta0 + nn) : 0.0;
  for (int32_t a = 0; a < D; ++a) {
    for (int32_t e = 0; e < D; ++e) {
      double sc = 0.0;
      for (int64_t s = 0; s < n; ++s) sc += (X[s * D + a] - xbar[a]) * (X[s * D + e] - xbar[e]);
      Winv_s[a * D + e] = W0inv[a * D + e] + sc + shrink * (mu0[a] - xbar[a]) * (mu0[e] - xbar[e]);
    }
    mu_s[a] = (beta0 * mu0[a] + nn * xbar[a]) / (beta0 + nn);
  }
  *beta_s = beta0 + nn;
  *nu_s = nu0 + nn;
  free(xbar);
}

/* Draw (mu, Lambda) from NW(mu_s, beta_s, W_s, nu_s) given W_s^{-1} (Winv_s) and the
 * variates: chi2[i] ~ chi-square with nu_s - i degrees of freedom (i = 0..D-1),
 * offd[k] ~ N(0,1) for the strict lower triangle in row order (k = i (i - 1) / 2 + j, j < i),
 * zmu[i] ~ N(0,1). Bartlett: W_s = F F^T (lower Cholesky), B lower triangular with
 * B_ii = sqrt(chi2[i]) and B_ij = offd, Lambda = (F B)(F B)^T; then with
 * beta_s Lambda = R R^T (lower Cholesky), mu = mu_s + R^{-T} zmu. Returns 0, or 1 if a
 * factorisation fails. */
int orc_nw_sample(int32_t D, const double *mu_s, double beta_s, const double *Winv_s,
                  const double *chi2, const double *offd, const double *zmu, double *mu_out,
                  double *Lambda_out) {
  const size_t DD = (size_t)D * D;
  double *R = (double *)malloc(sizeof(double) * DD);
  double *W = (double *)malloc(sizeof(double) * DD);
  double *Fm = (double *)malloc(sizeof(double) * DD);
  double *FB = (double *)malloc(sizeof(double) * DD);
  double *col = (double *)malloc(sizeof(double) * D);
  double *tmp = (double *)malloc(sizeof(double) * D);
  int st = 0;
  /* W_s = (W_s^{-1})^{-1}, column by column through the Cholesky factor of W_s^{-1} */
  if (chol_lower(D, Winv_s, R) != 0) st = 1;
  for (int32_t e = 0; e < D && st == 0; ++e) {
    for (int32_t a = 0; a < D; ++a) col[a] = a == e ? 1.0 : 0.0;
    solve_lower(D, R, col, tmp);
    solve_lower_t(D, R, tmp, col);
    for (int32_t a = 0; a < D; ++a) W[a * D + e] = col[a];
  }
  if (st == 0 && chol_lower(D, W, Fm) != 0) st = 1;
  if (st == 0) {
    /* F B, with B lower triangular */
    for (int32_t a = 0; a < D; ++a) {
      for (int32_t e = 0; e < D; ++e) {
        double t = 0.0;
        for (int32_t m = e; m <= a; ++m) {
          const double b = m == e ? sqrt(chi2[e]) : offd[(int64_t)m * (m - 1) / 2 + e];
          t += Fm[a * D + m] * b;
        }
        FB[a * D + e] = t;
      }
    }
    for (int32_t a = 0; a < D; ++a) {
      for (int32_t e = 0; e < D; ++e) {
        double t = 0.0;
        for (int32_t m = 0; m < D; ++m) t += FB[a * D + m] * FB[e * D + m];
        Lambda_out[a * D + e] = t;
      }
    }
    for (size_t q = 0; q < DD; ++q) W[q] = beta_s * Lambda_out[q];
    if (chol_lower(D, W, R) != 0) st = 1;
  }
  if (st == 0) {
    solve_lower_t(D, R, zmu, tmp);
    for (int32_t a = 0; a < D; ++a) mu_out[a] = mu_s[a] + tmp[a];
  }
  free(R); free(W); free(Fm); free(FB); free(col); free(tmp);
  return st;
}

/* ---- tensor ALS ------------------------------------------------------------------------ */

/* One mode's half-sweep of tensor ALS: for every row s, the ALS update (solve_one) with the
 * fixed vectors f_k = F1[idx1[k]] * F2[idx2[k]] (elementwise) of its ratings. Rows with no
 * ratings and flagged rows keep their previous X; flags as orc_half_sweep. */
int64_t orc_tensor_rows(int64_t n_rows, const int64_t *ptr, const int32_t *idx1,
                        const int32_t *idx2, const double *val, int32_t D, const double *F1,
                        const double *F2, double lambda, double *X, int8_t *flags, int nthreads) {
  set_threads(nthreads);
  int64_t maxdeg = 0;
  for (int64_t s = 0; s < n_rows; ++s) {
    if (ptr[s + 1] - ptr[s] > maxdeg) maxdeg = ptr[s + 1] - ptr[s];
  }
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *W = (double *)malloc(sizeof(double) * D * D);
    double *b = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
    double *Fs = (double *)malloc(sizeof(double) * D * (maxdeg > 0 ? maxdeg : 1));
    int32_t *seq = (int32_t *)malloc(sizeof(int32_t) * (maxdeg > 0 ? maxdeg : 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t s = 0; s < n_rows; ++s) {
      const int64_t n = ptr[s + 1] - ptr[s];
      for (int64_t q = 0; q < n; ++q) {
        const double *f1 = F1 + (int64_t)idx1[ptr[s] + q] * D;
        const double *f2 = F2 + (int64_t)idx2[ptr[s] + q] * D;
        for (int32_t a = 0; a < D; ++a) Fs[q * D + a] = f1[a] * f2[a];
        seq[q] = (int32_t)q;
      }
      int st = solve_one(D, n, seq, val + ptr[s], NULL, Fs, lambda, A, b, W, xs, X + s * D);
      if (flags) flags[s] = (int8_t)st;
      nflag += (st == 1);
    }
    free(A); free(W); free(b); free(xs); free(Fs); free(seq);
  }
  return nflag;
}

/* Sum over the rows' ratings of (r - sum_d X[s][d] F1[idx1][d] F2[idx2][d])^2, per row in
 * rating order and over rows in row order. */
double orc_tensor_sse(int64_t n_rows, const int64_t *ptr, const int32_t *idx1, const int32_t *idx2,
                      const double *val, int32_t D, const double *X, const double *F1,
                      const double *F2, int nthreads) {
  set_threads(nthreads);
  double *per = (double *)malloc(sizeof(double) * (n_rows > 0 ? n_rows : 1));
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t s = 0; s < n_rows; ++s) {
    double acc = 0.0;
    for (int64_t p = ptr[s]; p < ptr[s + 1]; ++p) {
      const double *f1 = F1 + (int64_t)idx1[p] * D;
      const double *f2 = F2 + (int64_t)idx2[p] * D;
      double pred = 0.0;
      for (int32_t a = 0; a < D; ++a) pred += X[s * D + a] * f1[a] * f2[a];
      const double e = val[p] - pred;
      acc += e * e;
    }
    per[s] = acc;
  }
  double total = 0.0;
  for (int64_t s = 0; s < n_rows; ++s) total += per[s];
  free(per);
  return total;
}

/* ---- BPTF: draws under the tensor model, the time factors' Markov chain ------------------ */
/*
 * Bayesian probabilistic tensor factorisation (the BPTF of Sec. 2.2 and Table 3, the
 * published sampler): the ratings are N(sum_d U_ud V_id T_td, 1/alpha); user and item rows
 * have the Normal-Wishart-governed priors of the matrix model; the time factors form a
 * Markov chain, T_0 ~ N(mu_T, Lambda_T^{-1}) and T_k ~ N(T_{k-1}, Lambda_T^{-1}) for
 * k >= 1, with (mu_T, Lambda_T) Normal-Wishart; and alpha has a one-dimensional Wishart
 * (scaled chi-square) prior.
 *
 * A row's full conditional is Gaussian with precision P = P0 + alpha sum_q f_q f_q^T and
 * P mean = h0 + alpha sum_q r_q f_q, where f_q is the elementwise product of the rating's
 * rows of the other two modes, and (P0, h0) come from the row's prior:
 *   user or item row:  P0 = Lambda,  h0 = Lambda mu;
 *   time bin k of K:   P0 = c_k Lambda_T with c_k = 2 if k < K - 1 (the bin is also the
 *                      condition of bin k + 1) and 1 for the last bin, and
 *                      h0 = Lambda_T (m_k + [k < K - 1] T_{k+1}) with m_k = mu_T for k = 0
 *                      and T_{k-1} otherwise.
 * The draw is x = L^{-T} (L^{-1} (P mean) + z) with P = L L^T.
 */

/* One draw as above. f_q = F1[idx1[q]] * F2[idx2[q]] over the row's n ratings; A, L, h, y
 * and xs are D x D / D scratch. Returns 0 (x_out written) or 1 (P not numerically SPD or a
 * non-finite result; x_out untouched). */
static int draw_tensor_row(int32_t D, int64_t n, const int32_t *idx1, const int32_t *idx2,
                           const double *val, const double *F1, const double *F2, double alpha,
                           const double *P0, const double *h0, const double *z, double *A,
                           double *L, double *h, double *y, double *xs, double *x_out) {
  for (int32_t a = 0; a < D * D; ++a) A[a] = 0.0;
  for (int32_t a = 0; a < D; ++a) h[a] = 0.0;
  for (int64_t q = 0; q < n; ++q) {
    const double *f1 = F1 + (int64_t)idx1[q] * D;
    const double *f2 = F2 + (int64_t)idx2[q] * D;
    for (int32_t a = 0; a < D; ++a) {
      const double fa = f1[a] * f2[a];
      for (int32_t e = 0; e < D; ++e) A[a * D + e] += fa * (f1[e] * f2[e]);
      h[a] += val[q] * fa;
    }
  }
  for (int32_t a = 0; a < D; ++a) {
    h[a] = alpha * h[a] + h0[a];
    for (int32_t e = 0; e < D; ++e) A[a * D + e] = alpha * A[a * D + e] + P0[a * D + e];
  }
  if (chol_lower(D, A, L) != 0) return 1;
  solve_lower(D, L, h, y);
  for (int32_t a = 0; a < D; ++a) y[a] += z[a];
  solve_lower_t(D, L, y, xs);
  for (int32_t a = 0; a < D; ++a) {
    if (!isfinite(xs[a])) return 1;
  }
  for (int32_t a = 0; a < D; ++a) x_out[a] = xs[a];
  return 0;
}

/* Conditional draw of every user (or item) row under the tensor model, prior N(mu,
 * Lambda^{-1}); z is n_rows x D. flags[s]: 0 drawn, 1 left unchanged. Returns the number of
 * flagged rows. */
int64_t orc_tensor_gibbs_rows(int64_t n_rows, const int64_t *ptr, const int32_t *idx1,
                              const int32_t *idx2, const double *val, int32_t D,
                              const double *F1, const double *F2, double alpha,
                              const double *Lambda, const double *mu, const double *z, double *X,
                              int8_t *flags, int nthreads) {
  set_threads(nthreads);
  double *h0 = (double *)malloc(sizeof(double) * D);
  for (int32_t a = 0; a < D; ++a) {
    double t = 0.0;
    for (int32_t e = 0; e < D; ++e) t += Lambda[a * D + e] * mu[e];
    h0[a] = t;
  }
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *L = (double *)malloc(sizeof(double) * D * D);
    double *h = (double *)malloc(sizeof(double) * D);
    double *y = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t s = 0; s < n_rows; ++s) {
      const int st = draw_tensor_row(D, ptr[s + 1] - ptr[s], idx1 + ptr[s], idx2 + ptr[s],
                                     val + ptr[s], F1, F2, alpha, Lambda, h0, z + s * D, A, L, h,
                                     y, xs, X + s * D);
      if (flags) flags[s] = (int8_t)st;
      nflag += st;
    }
    free(A); free(L); free(h); free(y); free(xs);
  }
  free(h0);
  return nflag;
}

/* Conditional draw of the time bins k = parity, parity + 2, ... (of K) given the bins of the
 * other parity; the other bins are read, never written. Bins of one parity are conditionally
 * independent given the rest (each conditional involves only the two neighbours), so one call
 * per parity, even then odd, is one Gibbs sweep over the chain. z is K x D (rows of the drawn
 * bins used). flags[k] for the drawn bins as above. Returns the number of flagged bins. */
int64_t orc_time_rows(int64_t K, const int64_t *ptr, const int32_t *idx1, const int32_t *idx2,
                      const double *val, int32_t D, const double *F1, const double *F2,
                      double alpha, const double *Lambda_T, const double *mu_T, const double *z,
                      int32_t parity, double *T, int8_t *flags, int nthreads) {
  set_threads(nthreads);
  int64_t nflag = 0;
#pragma omp parallel reduction(+ : nflag)
  {
    double *A = (double *)malloc(sizeof(double) * D * D);
    double *L = (double *)malloc(sizeof(double) * D * D);
    double *P0 = (double *)malloc(sizeof(double) * D * D);
    double *h = (double *)malloc(sizeof(double) * D);
    double *h0 = (double *)malloc(sizeof(double) * D);
    double *nb = (double *)malloc(sizeof(double) * D);
    double *y = (double *)malloc(sizeof(double) * D);
    double *xs = (double *)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 1)
    for (int64_t k = parity; k < K; k += 2) {
      const double ck = k < K - 1 ? 2.0 : 1.0;
      for (int32_t a = 0; a < D; ++a) {
        const double prev = k == 0 ? mu_T[a] : T[(k - 1) * D + a];
        const double next = k < K - 1 ? T[(k + 1) * D + a] : 0.0;
        nb[a] = prev + next;
      }
      for (int32_t a = 0; a < D; ++a) {
        double t = 0.0;
        for (int32_t e = 0; e < D; ++e) {
          t += Lambda_T[a * D + e] * nb[e];
          P0[a * D + e] = ck * Lambda_T[a * D + e];
        }
        h0[a] = t;
      }
      const int st = draw_tensor_row(D, ptr[k + 1] - ptr[k], idx1 + ptr[k], idx2 + ptr[k],
                                     val + ptr[k], F1, F2, alpha, P0, h0, z + k * D, A, L, h, y,
                                     xs, T + k * D);
      if (flags) flags[k] = (int8_t)st;
      nflag += st;
    }
    free(A); free(L); free(P0); free(h); free(h0); free(nb); free(y); free(xs);
  }
  return nflag;
}

/* Normal-Wishart posterior of (mu_T, Lambda_T) given the chain T (K x D, K >= 1) and the prior
 * (mu0, beta0, W0^{-1}, nu0): T_0 is one draw around mu_T and each step T_k - T_{k-1} one
 * zero-mean draw, so
 *   beta* = beta0 + 1,  nu* = nu0 + K,  mu0* = (beta0 mu0 + T_0) / (beta0 + 1),
 *   W*^{-1} = W0^{-1} + sum_{k>=1} (T_k - T_{k-1})(T_k - T_{k-1})^T
 *             + beta0 / (beta0 + 1) (T_0 - mu0)(T_0 - mu0)^T. */
void orc_time_posterior(int64_t K, int32_t D, const double *T, const double *mu0, double beta0,
                        const double *W0inv, double nu0, double *mu_s, double *Winv_s,
                        double *beta_s, double *nu_s) {
  const double w1 = beta0 / (beta0 + 1.0);
  for (int32_t a = 0; a < D; ++a) {
    for (int32_t e = 0; e < D; ++e) {
      double steps = 0.0;
      for (int64_t k = 1; k < K; ++k)
        steps += (T[k * D + a] - T[(k - 1) * D + a]) * (T[k * D + e] - T[(k - 1) * D + e]);
      Winv_s[a * D + e] = W0inv[a * D + e] + steps + w1 * (T[a] - mu0[a]) * (T[e] - mu0[e]);
    }
    mu_s[a] = (beta0 * mu0[a] + T[a]) / (beta0 + 1.0);
  }
  *beta_s = beta0 + 1.0;
  *nu_s = nu0 + (double)K;
}
