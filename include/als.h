/*
 * als.h -- C ABI of the MI355X (gfx950) alternating-least-squares half-sweep.
 *
 * The method (paper Sec. 2.2, "ALS and BPTF"): a sparse M x N matrix A of
 * observed ratings (users x items) is modelled as U V, with U (M x D) and V
 * (D x N). ALS alternates: with U held, every item column of V is a
 * least-squares fit; with V held, every user row of U is. A rating is
 * predicted by the inner product of its user's and its item's vectors. One
 * least-squares pass over one side is a "half-sweep":
 *
 *   for every row s of the solved side with n_s = |Omega_s| > 0 ratings,
 *     x_s = (sum_{j in Omega_s} f_j f_j^T + lambda * n_s * I)^{-1}
 *           * sum_{j in Omega_s} r_sj f_j,
 *
 * where f_j are the fixed side's rows. The per-update inversion
 * (Sec. 4.1) is done by Cholesky. The quality measure is RMSE (Sec. 4.1),
 * here the training RMSE over all stored ratings.
 *
 * Conventions
 *  - Layout: U is stored [n_users x D] and V is stored [n_items x D], both
 *    row-major fp32 (V transposed relative to the paper's D x N, so that one
 *    item's vector is contiguous).
 *  - The rating matrix is given once, as host CSR by user; every stored
 *    position is an observed rating, including explicit zeros.
 *  - Ownership: the library copies the CSR to the device and owns it, the
 *    device-built CSC, the row schedules and all workspace. The caller owns
 *    every factor buffer (device memory, e.g. torch tensors).
 *  - Execution: work is enqueued on the HIP stream given at creation. A call
 *    synchronises that stream only where stated (RMSE read-back, flag count).
 *  - Errors: every call returns an als_status; nothing is thrown across the
 *    ABI. als_last_error() gives a message for the last failing call.
 *  - Threading: calls on one context must not overlap.
 *  - Determinism: results are bitwise reproducible run to run (fixed
 *    reduction orders, no floating-point atomics).
 */
#ifndef ALS_MI355X_H
#define ALS_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct als_ctx als_ctx;

typedef enum {
  ALS_OK = 0,
  ALS_ERR_INVALID_ARG = 1,   /* bad pointer, size, D, lambda, side, aliasing */
  ALS_ERR_BAD_MATRIX = 2,    /* CSR fails validation (see als_create) */
  ALS_ERR_OUT_OF_MEMORY = 3, /* device or host allocation failed */
  ALS_ERR_HIP = 4,           /* a HIP runtime call failed (message has details) */
  ALS_ERR_NOT_SPD = 5        /* half-sweep completed; >= 1 row flagged and left unchanged */
} als_status;

typedef enum {
  ALS_ROWS_USERS = 0, /* solve U (rows of the CSR) with V fixed */
  ALS_ROWS_ITEMS = 1  /* solve V (rows of the CSC) with U fixed */
} als_side;

typedef enum {
  ALS_MODE_USERS = 0, /* tensor ALS: solve U with V and T fixed */
  ALS_MODE_ITEMS = 1, /* solve V with U and T fixed */
  ALS_MODE_TIME = 2   /* solve T (one row per time bin) with U and V fixed */
} als_mode;

/* Tunables of the degree-bucketed schedule. Zero fields select defaults. */
typedef struct {
  int32_t hub_threshold;   /* rows with more ratings are split into chunks (default 8192) */
  int32_t chunk;           /* ratings per chunk of a split row (default 4096) */
  int64_t workspace_bytes; /* cap on the partial-Gram workspace; larger half-sweeps run in
                              several batches (default 48 GiB) */
} als_tuning;

/*
 * Create a context for one rating matrix and one factor width D: the observed ratings
 * of paper Sec. 2.2 (matrix A, users x items; every stored position is observed, Sec. 3
 * rates on 0..100 with 0 a valid rating) and the width D of the factors U and V.
 *   n_users, n_items  matrix shape (M, N); each >= 1, and (max(M, N) + 1) * DP * 4
 *                     < 2^32 bytes with DP = 16 * ceil(D / 16) (the staged fixed side
 *                     is addressed with 32-bit offsets): up to 8.4M rows per side at
 *                     D = 128, 33.5M at D = 20.
 *   nnz               number of stored ratings; 0 <= nnz < 2^31.
 *   row_ptr           host int64[n_users + 1]: row_ptr[0] = 0, non-decreasing,
 *                     row_ptr[n_users] = nnz.
 *   col_idx           host int32[nnz]: item of each rating, in [0, n_items),
 *                     strictly increasing within each row (no duplicates).
 *   ratings           host uint8[nnz]: the rating values (0..255 accepted).
 *   D                 factor width, 1 <= D <= 128.
 *   hip_stream        hipStream_t to enqueue on (NULL = default stream).
 *   tuning            nullable; see als_tuning.
 * Validation failures return ALS_ERR_BAD_MATRIX or ALS_ERR_INVALID_ARG and
 * set *out = NULL. On success the host arrays may be freed by the caller.
 * The call builds the item-major layout (CSC) on the device and the per-side
 * row schedules; it synchronises the stream before returning.
 */
als_status als_create(als_ctx **out, int64_t n_users, int64_t n_items, int64_t nnz,
                      const int64_t *row_ptr, const int32_t *col_idx, const uint8_t *ratings,
                      int32_t D, void *hip_stream, const als_tuning *tuning);

/*
 * One half-sweep (paper Sec. 2.2). The pass that gathers each row's fixed
 * vectors also accumulates the squared residuals of the state entering the
 * half-sweep (out_factors' previous content against fixed_factors); that
 * training RMSE (Sec. 4.1) is read back with als_last_rmse_in.
 *   side           ALS_ROWS_USERS: fixed = V [n_items x D], out = U [n_users x D].
 *                  ALS_ROWS_ITEMS: fixed = U [n_users x D], out = V [n_items x D].
 *   fixed_factors  device fp32, row-major, read only.
 *   lambda         regularisation weight, finite and >= 0; the diagonal gets
 *                  lambda * n_s for a row with n_s ratings.
 *   out_factors    device fp32, row-major, must not overlap fixed_factors.
 *                  The caller pre-fills it with the previous iterate: rows with
 *                  no ratings and flagged rows (pivot <= 0 or non-finite in the
 *                  Cholesky) keep that content.
 *   rmse_out       host, nullable. If non-NULL the call synchronises the stream
 *                  and writes the training RMSE of the new state (out_factors
 *                  against fixed_factors over all ratings), and returns
 *                  ALS_ERR_NOT_SPD if any row was flagged.
 */
als_status als_half_sweep(als_ctx *ctx, als_side side, const float *fixed_factors, float lambda,
                          float *out_factors, double *rmse_out);

/*
 * Training RMSE of the state that entered the most recent half-sweep (for a
 * sweep items-then-users: the RMSE after the previous half-sweep).
 * Synchronises the stream. ALS_ERR_INVALID_ARG if no half-sweep has run.
 */
als_status als_last_rmse_in(als_ctx *ctx, double *rmse_in);

/*
 * Training RMSE of (U, V), the quality measure of paper Sec. 4.1 over the stored ratings,
 * with the inner-product prediction of Sec. 2.2:
 * sqrt(sum over stored ratings of (r - u_u . v_i)^2 / nnz).
 * U, V: device fp32 [n_users x D], [n_items x D]. Synchronises the stream.
 * An empty matrix gives 0.
 */
als_status als_rmse(als_ctx *ctx, const float *U, const float *V, double *rmse_out);

/* Rows flagged (not SPD / non-finite, so the Cholesky of the per-update inversion of
 * Sec. 4.1 failed) by the last half-sweep; synchronises the stream. Returns -1 for a NULL
 * context or a failed synchronisation. */
int64_t als_flagged_rows(const als_ctx *ctx);

/*
 * Copy the device-built CSC (rows ascending within each column) to host
 * buffers: col_ptr int64[n_items + 1], row_idx int32[nnz], ratings uint8[nnz].
 * Synchronises the stream.
 */
als_status als_get_csc(als_ctx *ctx, int64_t *col_ptr, int32_t *row_idx, uint8_t *ratings);

/*
 * Schedule statistics of one side, for tests and reports. out receives up to
 * n values in this order: rows with ratings, rows split into chunks, chunks,
 * batches, largest degree, workspace bytes per batch, bytes per workspace slot.
 */
als_status als_plan_stats(als_ctx *ctx, als_side side, int64_t *out, int32_t n);

/*
 * Optional per-phase timing with HIP events recorded on the context's stream
 * around each kernel launch (no synchronisation while enabled). Phases:
 * 0 = staging of the fixed side; 1 = gather kernels (D <= 20: the normal
 * equations of every row and chunk; D > 20: those of split-row chunks);
 * 2 = solve kernels (D <= 20: one row per lane; D > 20: the fused row kernel,
 * which also builds the normal equations of unsplit rows); 3 = new-state
 * residual pass; 4 = reductions. enable: 0 = off; 1 = every phase; 2 = only the
 * launches that build the normal equations (phase 1, and phase 2 above D = 20), so
 * that no event record sits between the other launches. Other values:
 * ALS_ERR_INVALID_ARG. Enabling (1 or 2) resets the totals; als_get_profile
 * synchronises the stream, folds the recorded events into the totals and returns the
 * summed milliseconds and launch count of one phase.
 */
als_status als_set_profiling(als_ctx *ctx, int32_t enable);
als_status als_get_profile(als_ctx *ctx, int32_t phase, double *total_ms, int64_t *launches);

/*
 * Weighted ALS (wALS: named beside ALS in the paper's Sec. 2 and Sec. 4, which do not
 * define its weighting). weights: host array of nnz floats, one non-negative finite
 * weight c per stored rating in CSR order (the order of col_idx / ratings at create);
 * the library copies it to the device in both orders (8 bytes per rating). Later
 * half-sweeps solve x_s = (sum_j c_sj f_j f_j^T + lambda n_s I)^{-1} sum_j c_sj r_sj f_j
 * (the regulariser keeps the count n_s, so unit weights give plain ALS exactly); the
 * RMSE stays the unweighted training RMSE. NULL detaches the weights. Errors:
 * ALS_ERR_INVALID_ARG for a negative or non-finite weight (nothing changes),
 * ALS_ERR_OUT_OF_MEMORY, ALS_ERR_HIP. Synchronises the context's stream.
 */
als_status als_set_weights(als_ctx *ctx, const float *weights);

/*
 * Optional phase clocks of the fused row kernel (widths D > 20, which build the
 * normal equations and factor them in one kernel, Sec. 2.2). While enabled, every
 * row records the wavefront clock cycles spent before its factorisation begins
 * (gather, Gram, right-hand side and residuals, or the sum of a split row's chunk
 * partials) and from there to its end (factorisation, solves, write), and each
 * half-sweep adds them up per side; this costs one stream synchronisation per
 * half-sweep and leaves the results unchanged. Enabling allocates 16 bytes per row
 * of the larger side on first use and resets the totals. als_get_phase_cycles
 * returns a side's totals (zero for D <= 20, whose Gram kernel is separate).
 */
als_status als_set_phase_timing(als_ctx *ctx, int32_t enable);
als_status als_get_phase_cycles(als_ctx *ctx, als_side side, double *gram_cycles,
                                double *solve_cycles);

/*
 * Held-out prediction (paper Sec. 2.2: a prediction is the dot product of the user's
 * and the item's vector) for n_pairs (user, item) pairs:
 *   pred[p] = U[users[p], :] . V[items[p], :]   (fp32, features summed in order).
 *   U, V          device fp32 [n_users x D], [n_items x D], 16-byte aligned.
 *   users, items  device int32[n_pairs]; a pair with an index outside the tables gets
 *                 pred = NaN and reads nothing.
 *   pred          device fp32[n_pairs], caller-owned, overlapping none of the inputs.
 * Enqueued on the context's stream without synchronisation. n_pairs = 0 does nothing;
 * n_pairs above (2^31 - 1) * 32 is ALS_ERR_INVALID_ARG.
 */
als_status als_predict(als_ctx *ctx, const float *U, const float *V, int64_t n_pairs,
                       const int32_t *users, const int32_t *items, float *pred);

/*
 * Register a validation set (Sec. 4.1 reports RMSE on ratings held out of training):
 * host arrays of n_pairs users, items and ratings. Every index is checked against the
 * matrix shape (ALS_ERR_INVALID_ARG, nothing registered). The library copies the pairs
 * to the device, grouped by user (stable, so the caller's order within a user stays),
 * and replaces any earlier set; n_pairs = 0 registers an empty set. Duplicates and
 * pairs that are also training ratings are allowed. Synchronises the stream.
 */
als_status als_set_holdout(als_ctx *ctx, int64_t n_pairs, const int32_t *users,
                           const int32_t *items, const uint8_t *ratings);

/*
 * Validation RMSE of (U, V) on the registered pairs:
 * sqrt(sum over pairs of (r - u_u . v_i)^2 / n_pairs), squared errors summed in fp64 in a
 * fixed order (bitwise reproducible). 0 for an empty set; ALS_ERR_INVALID_ARG when no set
 * is registered. U, V as for als_predict. Synchronises the stream.
 */
als_status als_holdout_rmse(als_ctx *ctx, const float *U, const float *V, double *rmse_out);

/*
 * Validation RMSE of (U, V) on caller-provided device pairs, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and fixed summation order as als_holdout_rmse,
 * with no registration and no allocation. Its scratch (per-block sums, the reduction's
 * partials and the total) is a fixed array of 4 MiB in device memory that every GPU the
 * library runs on holds until the process ends; the call neither allocates nor frees.
 *   users, items, ratings  device int32[n_pairs], int32[n_pairs], uint8[n_pairs], read only;
 *                          a pair with an index outside the tables makes the result NaN.
 *                          Pairs grouped by user (as als_set_holdout stores them) give the
 *                          registered set's result bit for bit.
 *   n_pairs                0 .. 16,000,000 (ALS_ERR_INVALID_ARG above: the scratch's limit);
 *                          0 gives 0.
 *   U, V, rmse_out         as for als_holdout_rmse. Synchronises the context's stream.
 * All calls on one GPU share its scratch array, whatever their context: calls that
 * overlap on one GPU (other host threads, other streams) race and must be serialised by
 * the caller.
 */
als_status als_pair_rmse_noalloc(als_ctx *ctx, const float *U, const float *V, int64_t n_pairs,
                                 const int32_t *users, const int32_t *items,
                                 const uint8_t *ratings, double *rmse_out);

/*
 * Bayesian factorisation (BPTF, paper Sec. 2.2, which pairs the least-squares update with
 * draws of the factor priors' parameters), as the published BPMF / BPTF Gibbs sampler: ratings are
 * Gaussian with precision alpha around u . v; each row of a side has the prior
 * N(mu, Lambda^{-1}); (mu, Lambda) has the Normal-Wishart hyperprior NW(mu0, beta0, W0, nu0).
 * One Gibbs step for a side: als_sample_hyper draws (mu, Lambda) given the side's rows,
 * then als_gibbs_half_sweep draws every row given the other side. Every random variate
 * is an input (device memory), so a step is a deterministic function of them.
 *
 * als_set_nw_prior: the hyperprior of one side (host arrays, copied): mu0[D], beta0 >= 0,
 * W0_inv[D x D] row-major, finite and symmetric (the inverse of the Wishart scale W0),
 * nu0 > D - 1. ALS_ERR_INVALID_ARG otherwise. Synchronises the stream.
 */
als_status als_set_nw_prior(als_ctx *ctx, als_side side, const double *mu0, double beta0,
                            const double *W0_inv, double nu0);

/*
 * Draw the side's hyperparameters from their Normal-Wishart posterior given its n rows
 * X (device fp32 [n x D], 16-byte aligned; n = n_users or n_items):
 *   beta* = beta0 + n, nu* = nu0 + n, mu0* = (beta0 mu0 + n xbar) / beta*,
 *   W*^{-1} = W0^{-1} + sum_s (x_s - xbar)(x_s - xbar)^T + beta0 n / beta* (mu0 - xbar)(mu0 - xbar)^T;
 * Bartlett's construction: W* = F F^T (lower Cholesky), B lower triangular with
 * B_ii = sqrt(chi2[i]) and B_ij = offdiag[i (i - 1) / 2 + j] (j < i), Lambda = (F B)(F B)^T;
 * then mu = mu0* + R^{-T} z_mu with beta* Lambda = R R^T.
 *   chi2      device fp64[D], chi2[i] drawn from the chi-square law with nu* - i degrees
 *             of freedom (i = 0 .. D-1);
 *   offdiag   device fp64[D (D - 1) / 2] standard normals (may be NULL when D = 1);
 *   z_mu      device fp64[D] standard normals;
 *   mu_out, Lambda_out  device fp64[D], [D x D], caller-owned.
 * Everything runs in fp64 on the device, enqueued without synchronisation. status_out
 * (host, nullable): if non-NULL the call synchronises and stores 0, or 1 when a
 * factorisation failed (then the return is ALS_ERR_NOT_SPD). ALS_ERR_INVALID_ARG when no
 * prior was set for the side.
 */
als_status als_sample_hyper(als_ctx *ctx, als_side side, const float *X, const double *chi2,
                            const double *offdiag, const double *z_mu, double *mu_out,
                            double *Lambda_out, int32_t *status_out);

/*
 * Gibbs half-sweep: every row s of the side drawn from its Gaussian conditional
 *   Lambda* = Lambda + alpha sum_j f_j f_j^T,  mu* = Lambda*^{-1} (alpha sum_j r_sj f_j + Lambda mu),
 *   x_s = mu* + L*^{-T} z_s  (Lambda* = L* L*^T),
 * with the same gather, Gram and factorisation kernels as als_half_sweep (the system is
 * solved as (G + Lambda / alpha) with z_s / sqrt(alpha) added before the back
 * substitution). Rows without ratings are drawn from the prior, x_s = mu + L^{-T} z_s
 * (Lambda = L L^T).
 *   alpha          rating precision, finite and > 0.
 *   Lambda, mu     device fp64 [D x D] (symmetric positive definite), [D] (e.g. the
 *                  outputs of als_sample_hyper).
 *   z              device fp32 [n_rows x D] standard normals, one row per row of the side.
 *   fixed_factors, out_factors, rmse_out: as for als_half_sweep (flagged rows, whose
 *                  Lambda* is not numerically SPD, keep their previous value).
 * The context must have no rating weights attached (ALS_ERR_INVALID_ARG).
 */
als_status als_gibbs_half_sweep(als_ctx *ctx, als_side side, const float *fixed_factors,
                                float alpha, const double *Lambda, const double *mu,
                                const float *z, float *out_factors, double *rmse_out);

/*
 * Tensor ALS (paper Sec. 2.2: the ALS model extended to the tensor case, with the time of
 * each rating; the data's ratings fall into time bins, Sec. 1). Every rating gets a time
 * bin t; the prediction is sum_d U[u][d] V[i][d] T[t][d] with T [n_bins x D] row-major fp32.
 * A mode's half-sweep is the ALS update of that mode's rows, whose fixed vectors are the
 * elementwise products of the other two modes' rows (V[i] * T[t] for a user, U[u] * T[t]
 * for an item, U[u] * V[i] for a time bin), with the same regulariser lambda * n_s.
 *
 * als_set_time_bins: bins = host int32[nnz], the time bin of every rating in CSR order
 * (the order of col_idx at create), each in [0, n_bins). The library keeps them on the
 * device in user, item and time-bin order (the last built by a stable counting sort on
 * the host, about 13 bytes per rating of host memory while it runs) and schedules the
 * time-bin rows like the other sides. Replaces an earlier set; ALS_ERR_INVALID_ARG for a
 * bin out of range (nothing changes). Synchronises the stream.
 */
als_status als_set_time_bins(als_ctx *ctx, int32_t n_bins, const int32_t *bins);

/*
 * One mode's half-sweep of tensor ALS: the rows of the mode's factor (U, V or T, device fp32,
 * 16-byte aligned, pairwise non-overlapping) are overwritten with their regularised
 * least-squares solutions given the other two (rows without ratings and flagged rows keep
 * their values). The gather of the same pass yields the squared residuals of the entering
 * state (als_last_rmse_in); rmse_out (host, nullable) as for als_half_sweep, over the
 * three-way predictions. ALS_ERR_INVALID_ARG without time bins or with weights attached.
 */
als_status als_tensor_half_sweep(als_ctx *ctx, als_mode mode, float *U, float *V, float *T,
                                 float lambda, double *rmse_out);

/* Training RMSE of the three-way predictions over all stored ratings; synchronises. */
als_status als_tensor_rmse(als_ctx *ctx, const float *U, const float *V, const float *T,
                           double *rmse_out);

/*
 * BPTF, the Bayesian tensor factorisation of paper Sec. 2.2 and Table 3, as the published
 * Gibbs sampler: the ratings are N(sum_d U[u][d] V[i][d] T[t][d], 1 / alpha); user and
 * item rows have the Normal-Wishart-governed priors N(mu, Lambda^{-1}) of the Gibbs
 * half-sweep; the time factors form a Markov chain, T[0] ~ N(mu_T, Lambda_T^{-1}) and
 * T[k] ~ N(T[k-1], Lambda_T^{-1}), with (mu_T, Lambda_T) Normal-Wishart; and alpha has a
 * one-dimensional Wishart prior W(w0, nu0) (w0 times a chi-square with nu0 degrees of
 * freedom). One iteration: als_tensor_sample_alpha; the hyperparameters of the items and
 * users (als_sample_hyper on V and U) and of the chain (als_sample_time_hyper); then
 * als_tensor_gibbs_half_sweep for the items, the users and the time bins.
 *
 * als_set_time_nw_prior: the chain's Normal-Wishart hyperprior, arguments as for
 * als_set_nw_prior.
 */
als_status als_set_time_nw_prior(als_ctx *ctx, const double *mu0, double beta0,
                                 const double *W0_inv, double nu0);

/*
 * Draw (mu_T, Lambda_T) from the chain's Normal-Wishart posterior given T (device fp32
 * [n_bins x D]): T[0] is one draw around mu_T and every step T[k] - T[k-1] a zero-mean
 * draw, so beta* = beta0 + 1, nu* = nu0 + n_bins, mu0* = (beta0 mu0 + T[0]) / beta*, and
 * W*^{-1} = W0^{-1} + sum_{k>=1} (T[k] - T[k-1])(T[k] - T[k-1])^T
 *           + beta0 / beta* (T[0] - mu0)(T[0] - mu0)^T;
 * then Bartlett's draw with the variates, all as for als_sample_hyper (chi2[i] with
 * nu* - i degrees of freedom). The steps are differenced in fp64. ALS_ERR_INVALID_ARG
 * without time bins or without a chain prior.
 */
als_status als_sample_time_hyper(als_ctx *ctx, const float *T, const double *chi2,
                                 const double *offdiag, const double *z_mu, double *mu_out,
                                 double *Lambda_out, int32_t *status_out);

/*
 * One mode of the BPTF Gibbs step: every row of the mode's factor (buffers as for
 * als_tensor_half_sweep) drawn from its Gaussian conditional given the other two modes,
 * with the fixed vectors of als_tensor_half_sweep and precision
 * P = P0 + alpha sum f f^T, mean P^{-1} (h0 + alpha sum r f), x = mean + L^{-T} z
 * (P = L L^T):
 *   ALS_MODE_USERS / ALS_MODE_ITEMS: P0 = Lambda, h0 = Lambda mu (Lambda, mu: device fp64,
 *     e.g. from als_sample_hyper); rows without ratings are drawn from that prior.
 *   ALS_MODE_TIME: Lambda, mu are the chain's (mu_T, Lambda_T); bin k has
 *     P0 = 2 Lambda_T (Lambda_T for the last bin) and
 *     h0 = Lambda_T (m_k + T[k+1]) with m_0 = mu_T, m_k = T[k-1], and no T[k+1] term for
 *     the last bin. The even bins are drawn first, given the odd ones, then the odd bins
 *     given the new even ones: the bins of one parity are conditionally independent, so
 *     this is one Gibbs sweep over the chain. Bins without ratings are drawn from their
 *     conditional in the same kernels.
 *   alpha   rating precision, finite and > 0.
 *   z       device fp32 [rows of the mode x D] standard normals.
 * rmse_out (host, nullable): as for als_tensor_half_sweep. Flagged rows keep their values.
 */
als_status als_tensor_gibbs_half_sweep(als_ctx *ctx, als_mode mode, float *U, float *V, float *T,
                                       float alpha, const double *Lambda, const double *mu,
                                       const float *z, double *rmse_out);

/*
 * Draw the rating precision from its posterior given the three factors: with the sum of
 * squared residuals sse over the stored ratings (computed on the device, fp64 sums),
 * alpha = chi2 / (1 / w0 + sse), where chi2 (host) is drawn from the chi-square law with
 * nu0 + nnz degrees of freedom. Synchronises; *alpha_out (host).
 */
als_status als_tensor_sample_alpha(als_ctx *ctx, const float *U, const float *V, const float *T,
                                   double w0, double chi2, double *alpha_out);

/* Release the context of als_create (the rating matrix of paper Sec. 2.2, its device
 * layouts, schedules and workspace) after synchronising its stream; NULL is ignored.
 * Caller-owned factor buffers are untouched. */
void als_destroy(als_ctx *ctx);

/* Text of a status code. Error reporting of this interface; no passage of the paper
 * defines it. The string is static. */
const char *als_status_str(als_status s);

/* Message of the last failing call on ctx (or of the last failed
 * als_create when ctx is NULL); valid until the next call on ctx. Error reporting of
 * this interface; no passage of the paper defines it. */
const char *als_last_error(const als_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* ALS_MI355X_H */
