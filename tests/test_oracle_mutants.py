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
    ("pair_error_sign", "const double e = r[p] - pred[p];", "const double e = r[p] + pred[p];"),
    ("pair_sse_first_dropped", "for (int64_t p = 0; p < n; ++p) {\n    const double e",
     "for (int64_t p = 1; p < n; ++p) {\n    const double e"),
]

PIN_TESTS = [
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
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", str(so), str(path), "-lm"])
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
