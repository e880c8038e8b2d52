"""The oracle pins must be sensitive: plant plausible mistakes in a copy of the
oracle's C source (on the CPU only), rebuild it, and check that the pins catch
every one of them."""
import ctypes
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins
from tests import test_oracle_weighted_pins as wpins
from tests import test_oracle_predict_pins as qpins
from tests import test_oracle_bayes_pins as bpins
from tests import test_oracle_tensor_pins as tpins
from tests import test_oracle_bptf_pins as btpins

SRC = os.path.join(os.path.dirname(oracle.__file__), "als_oracle.c")

# (name, original text, mutated text)
MUTANTS = [
    ("unweighted_lambda", "A[a * D + a] += lambda * (double)n;", "A[a * D + a] += lambda;"),
    ("rhs_without_rating", "b[a] += r * cf;", "b[a] += cf;"),
    ("first_rating_dropped", "for (int64_t k = 0; k < n; ++k) {", "for (int64_t k = 1; k < n; ++k) {"),
    ("backsolve_transposed", "s -= W[m * D + i] * x[m];", "s -= W[i * D + m] * x[m];"),
    ("cholesky_sign", "s -= W[i * D + m] * W[j * D + m];", "s += W[i * D + m] * W[j * D + m];"),
    ("forward_solve_no_update", "s -= W[i * D + m] * y[m];", "s -= 0.0 * y[m];"),
    ("prediction_wrong_index", "pred += x[a] * f[a];", "pred += x[a] * f[0];"),
    ("transpose_rows_reversed", "for (int64_t r = 0; r < n_rows; ++r) {\n    for (int64_t p = ptr[r];",
     "for (int64_t r = n_rows - 1; r >= 0; --r) {\n    for (int64_t p = ptr[r];"),
    ("norm_unweighted", "total += (double)(ptr[s + 1] - ptr[s]) * q;", "total += q;"),
    ("zero_degree_overwritten", "if (n == 0) return 2;", "if (n < 0) return 2;"),
    ("weight_squared", "const double cf = wt ? wt[k] * f[a] : f[a];",
     "const double cf = wt ? wt[k] * wt[k] * f[a] : f[a];"),
    ("weight_ignored_in_gram", "for (int32_t e = 0; e < D; ++e) A[a * D + e] += cf * f[e];",
     "for (int32_t e = 0; e < D; ++e) A[a * D + e] += f[a] * f[e];"),
    ("weight_ignored_in_rhs", "b[a] += r * cf;", "b[a] += r * f[a];"),
    ("weight_offset_wrong_row", "wt ? wt + ptr[s] : NULL, F, lambda, A, b, W, xs, X + s * D);",
     "wt ? wt + ptr[s] + 1 : NULL, F, lambda, A, b, W, xs, X + s * D);"),
    ("weighted_sse_unweighted", "acc += wt ? wt[p] * (e * e) : e * e;", "acc += e * e;"),
    ("predict_user_row_from_item", "const double *u = U + (int64_t)users[p] * D;",
     "const double *u = U + (int64_t)items[p] * D;"),
    ("predict_last_feature_dropped", "for (int32_t a = 0; a < D; ++a) dot += u[a] * v[a];",
     "for (int32_t a = 0; a + 1 < D; ++a) dot += u[a] * v[a];"),
    ("gibbs_prior_mean_dropped", "h[a] = alpha * h[a] + lm;", "h[a] = alpha * h[a];"),
    ("gibbs_gram_without_alpha",
     "for (int32_t e = 0; e < D; ++e) A[a * D + e] = alpha * A[a * D + e] + Lambda[a * D + e];",
     "for (int32_t e = 0; e < D; ++e) A[a * D + e] = A[a * D + e] + Lambda[a * D + e];"),
    ("gibbs_noise_halved", "for (int32_t a = 0; a < D; ++a) y[a] += z[s * D + a];",
     "for (int32_t a = 0; a < D; ++a) y[a] += 0.5 * z[s * D + a];"),
    ("gibbs_noise_lower_solve", "solve_lower_t(D, L, y, x);\n        for (int32_t a = 0; a < D; ++a) {\n          if (!isfinite",
     "solve_lower_t(D, L, y, x);\n        solve_lower(D, L, y, x);\n        for (int32_t a = 0; a < D; ++a) {\n          if (!isfinite"),
    ("nw_shrinkage_dropped",
     "+ sc + shrink * (mu0[a] - xbar[a]) * (mu0[e] - xbar[e]);", "+ sc;"),
    ("nw_mean_unshrunk", "mu_s[a] = (beta0 * mu0[a] + nn * xbar[a]) / (beta0 + nn);",
     "mu_s[a] = xbar[a];"),
    ("nw_wishart_transposed_product", "for (int32_t m = 0; m < D; ++m) t += FB[a * D + m] * FB[e * D + m];",
     "for (int32_t m = 0; m < D; ++m) t += FB[m * D + a] * FB[m * D + e];"),
    ("nw_bartlett_diagonal_not_rooted", "const double b = m == e ? sqrt(chi2[e]) :",
     "const double b = m == e ? chi2[e] :"),
    ("nw_mean_noise_wrong_solve", "solve_lower_t(D, R, zmu, tmp);", "solve_lower(D, R, zmu, tmp);"),
    ("tensor_product_dropped", "for (int32_t a = 0; a < D; ++a) Fs[q * D + a] = f1[a] * f2[a];",
     "for (int32_t a = 0; a < D; ++a) Fs[q * D + a] = f1[a];"),
    ("tensor_second_index_wrong", "const double *f2 = F2 + (int64_t)idx2[ptr[s] + q] * D;",
     "const double *f2 = F2 + (int64_t)idx2[ptr[s]] * D;"),
    ("tensor_sse_without_time", "for (int32_t a = 0; a < D; ++a) pred += X[s * D + a] * f1[a] * f2[a];",
     "for (int32_t a = 0; a < D; ++a) pred += X[s * D + a] * f1[a];"),
    ("bptf_second_factor_dropped", "const double fa = f1[a] * f2[a];", "const double fa = f1[a];"),
    ("bptf_prior_linear_term_dropped", "h[a] = alpha * h[a] + h0[a];", "h[a] = alpha * h[a];"),
    ("bptf_noise_not_added", "for (int32_t a = 0; a < D; ++a) y[a] += z[a];",
     "for (int32_t a = 0; a < D; ++a) y[a] += 0.0 * z[a];"),
    ("time_last_bin_doubled", "const double ck = k < K - 1 ? 2.0 : 1.0;", "const double ck = 2.0;"),
    ("time_interior_bin_single", "const double ck = k < K - 1 ? 2.0 : 1.0;",
     "const double ck = k < K - 1 ? 1.0 : 1.0;"),
    ("time_first_bin_without_mean", "const double prev = k == 0 ? mu_T[a] : T[(k - 1) * D + a];",
     "const double prev = k == 0 ? 0.0 : T[(k - 1) * D + a];"),
    ("time_next_neighbour_dropped", "const double next = k < K - 1 ? T[(k + 1) * D + a] : 0.0;",
     "const double next = 0.0;"),
    ("time_parity_stride_one", "for (int64_t k = parity; k < K; k += 2) {",
     "for (int64_t k = parity; k < K; k += 1) {"),
    ("time_posterior_steps_not_differenced",
     "steps += (T[k * D + a] - T[(k - 1) * D + a]) * (T[k * D + e] - T[(k - 1) * D + e]);",
     "steps += T[k * D + a] * T[k * D + e];"),
    ("time_posterior_first_step_dropped", "for (int64_t k = 1; k < K; ++k)\n        steps +=",
     "for (int64_t k = 2; k < K; ++k)\n        steps +="),
    ("time_posterior_shrink_dropped", "+ steps + w1 * (T[a] - mu0[a]) * (T[e] - mu0[e]);", "+ steps;"),
    ("time_posterior_mean_unshrunk", "mu_s[a] = (beta0 * mu0[a] + T[a]) / (beta0 + 1.0);",
     "mu_s[a] = T[a];"),
    ("time_posterior_dof_per_row", "*nu_s = nu0 + (double)K;", "*nu_s = nu0 + 1.0;"),
    ("pair_error_sign", "const double e = r[p] - pred[p];", "const double e = r[p] + pred[p];"),
    ("pair_sse_first_dropped", "for (int64_t p = 0; p < n; ++p) {\n    const double e",
     "for (int64_t p = 1; p < n; ++p) {\n    const double e"),
]

PIN_TESTS = [
    lambda: btpins.test_bt1_unit_time_factors_give_the_matrix_draw(4),
    btpins.test_bt2_tensor_row_uses_the_elementwise_product,
    lambda: btpins.test_bt3_bins_are_the_joint_gaussians_conditionals(5, 3),
    lambda: btpins.test_bt3_bins_are_the_joint_gaussians_conditionals(8, 2),
    btpins.test_bt4_single_bin_chain_is_the_matrix_prior_draw,
    btpins.test_bt5_empty_interior_bin_without_noise_is_the_neighbours_mean,
    lambda: btpins.test_bt6_time_posterior_is_conjugate(4, 2),
    lambda: btpins.test_bt6_time_posterior_is_conjugate(9, 3),
    btpins.test_bt7_one_bin_posterior_is_the_one_row_posterior,
    tpins.test_t1_unit_time_factors_give_matrix_als,
    lambda: tpins.test_t2_matches_least_squares_on_the_product_design(3),
    tpins.test_t3_objective_gradient_vanishes_after_each_mode,
    tpins.test_t4_objective_never_increases,
    tpins.test_t6_unit_time_factors_give_the_training_sse,
    lambda: bpins.test_b1_zero_noise_isotropic_prior_is_ridge(3),
    bpins.test_b2_zero_noise_is_the_posterior_mode,
    bpins.test_b3_noise_has_the_conditional_covariance,
    bpins.test_b4_row_without_ratings_is_a_prior_draw,
    bpins.test_b6_conjugate_update_batch_equals_sequential,
    bpins.test_b7_flat_prior_gives_the_sample_scatter,
    bpins.test_b8_unit_variates_give_the_scale_matrix,
    bpins.test_b9_mean_draw_has_covariance_of_beta_lambda_inverse,
    bpins.test_b10_wishart_moments,
    qpins.test_q1_golden_predictions,
    qpins.test_q2_dense_pairs_are_the_matrix_product,
    qpins.test_q3_stored_positions_give_the_training_sse,
    wpins.test_w1_unit_weights_are_plain_als,
    lambda: wpins.test_w2_matches_weighted_lstsq(3),
    wpins.test_w3_weighted_gradient_zero,
    wpins.test_w5_integer_weight_is_repeated_rating,
    wpins.test_w7_single_rating_closed_form,
    wpins.test_w9_weighted_sse,
    pins.test_golden_worked_solves,
    pins.test_golden_worked_rmse,
    lambda: pins.test_brute_force_rational(3, 5),
    lambda: pins.test_p1_matches_lstsq(3),
    pins.test_p2_gradient_zero,
    pins.test_p4_single_rating_sherman_morrison,
    pins.test_p4_one_factor,
    pins.test_p4_orthogonal_rows,
    pins.test_p5_dense_soft_threshold,
    pins.test_p7_symmetry,
    pins.test_p10_transpose,
    pins.test_p11_rmse_gram_identity,
    pins.test_empty_row_unchanged_and_zero_ratings_counted,
]


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, f"mutation anchor not unique for {name}"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(orig, mut))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", *oracle.CFLAGS, "-shared", "-fPIC", "-o", str(so), str(path), "-lm"])
    saved = oracle._lib
    oracle._lib = oracle._configure(ctypes.CDLL(str(so)))
    caught = []
    try:
        for t in PIN_TESTS:
            try:
                t()
            except (AssertionError, ValueError, StopIteration, IndexError, ZeroDivisionError):
                caught.append(getattr(t, "__name__", "lambda"))
    finally:
        oracle._lib = saved
    assert caught, f"no pin caught mutant {name}"
