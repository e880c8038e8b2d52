"""Pins of the oracle's tensor ALS (the ALS model with each rating's time bin: prediction
sum_d U_ud V_id T_td, each mode solved with the elementwise products of the other two
modes' rows as its fixed vectors).

Facts that do not come from the oracle: unit time factors reduce a mode update to the
matrix ALS update (itself pinned), numpy least squares on the product design, the
stationarity of the objective computed from the ratings, the monotone objective over
mode updates, exact recovery of noise-free low-rank tensors, and the training SSE with
unit time factors. Shapes keep every index inside every table, so a planted index mix-up
gives wrong values rather than an out-of-range read.
"""
import numpy as np
import pytest

import oracle
import workload
from tests.test_oracle_pins import rand_csr


def tensor_case(seed, M=30, N=24, n_bins=40, D=4, density=0.35):
    rng = np.random.default_rng(seed)
    ptr, col, val = rand_csr(rng, M, N, density, min_deg=2)
    bins = rng.integers(0, n_bins, size=col.size).astype(np.int32)
    U = rng.normal(0, 0.5, size=(M, D))
    V = rng.normal(0, 0.5, size=(N, D))
    T = rng.normal(1.0, 0.3, size=(n_bins, D))
    return rng, ptr, col, bins, val, U, V, T


def test_t1_unit_time_factors_give_matrix_als():
    _, ptr, col, bins, val, U, V, T = tensor_case(60)
    lam = 0.065
    ones = np.ones_like(T)
    Xt, ft = oracle.tensor_rows(ptr, col, bins, val, V, ones, lam, np.zeros_like(U))
    Xa, fa = oracle.half_sweep(ptr, col, val, V, lam, np.zeros_like(U))
    assert np.array_equal(Xt, Xa) and np.array_equal(ft, fa)


@pytest.mark.parametrize("D", [1, 3, 5])
def test_t2_matches_least_squares_on_the_product_design(D):
    _, ptr, col, bins, val, U, V, T = tensor_case(61 + D, D=D)
    lam = 0.3
    X, fl = oracle.tensor_rows(ptr, col, bins, val, V, T, lam, np.zeros_like(U))
    assert not fl.any()
    for s in range(ptr.size - 1):
        k = slice(ptr[s], ptr[s + 1])
        Fs = V[col[k]] * T[bins[k]]
        n = ptr[s + 1] - ptr[s]
        A = np.vstack([Fs, np.sqrt(lam * n) * np.eye(D)])
        y = np.concatenate([val[k], np.zeros(D)])
        want = np.linalg.lstsq(A, y, rcond=None)[0]
        np.testing.assert_allclose(X[s], want, rtol=1e-10, atol=1e-10)


def test_t3_objective_gradient_vanishes_after_each_mode():
    _, ptr, col, bins, val, U, V, T = tensor_case(64)
    M, N, n_bins = U.shape[0], V.shape[0], T.shape[0]
    lam = 0.1
    t = oracle.TensorTrajectory(M, N, n_bins, ptr, col, bins, val, U, V, T, lam)
    # mode, its grouping of the ratings, its factor, the two fixed factors
    for mode, groups, Xn, F1, F2 in (("items", "by_item", "V", "U", "T"),
                                     ("users", "by_user", "U", "V", "T"),
                                     ("bins", "by_bin", "T", "U", "V")):
        t.step(mode)
        X = getattr(t, Xn)
        p, i1, i2, v = getattr(t, groups)
        A1, A2 = getattr(t, F1), getattr(t, F2)
        for s in range(p.size - 1):
            k = slice(p[s], p[s + 1])
            if p[s + 1] == p[s]:
                continue
            f = A1[i1[k]] * A2[i2[k]]
            g = f.T @ (v[k] - f @ X[s]) - lam * (p[s + 1] - p[s]) * X[s]
            assert np.linalg.norm(g) <= 1e-9 * (np.abs(f.T @ v[k]).sum() + 1)


def test_t4_objective_never_increases():
    _, ptr, col, bins, val, U, V, T = tensor_case(65, M=40, N=30, n_bins=12)
    lam = 0.05
    t = oracle.TensorTrajectory(U.shape[0], V.shape[0], T.shape[0], ptr, col, bins, val, U, V,
                                T, lam)

    def objective():
        p, i1, i2, v = t.by_user
        reg = lam * sum(np.dot(np.diff(g[0]), (X * X).sum(1))
                        for g, X in ((t.by_user, t.U), (t.by_item, t.V), (t.by_bin, t.T)))
        return oracle.tensor_sse(p, i1, i2, v, t.U, t.V, t.T) + reg

    last = objective()
    for _ in range(4):
        for mode in ("items", "users", "bins"):
            t.step(mode)
            now = objective()
            assert now <= last * (1 + 1e-12)
            last = now


def test_t5_noise_free_low_rank_tensor_is_recovered():
    rng = np.random.default_rng(66)
    M, N, n_bins, k = 50, 40, 10, 2
    Us, Vs, Ts = rng.normal(size=(M, k)), rng.normal(size=(N, k)), rng.normal(1, 0.5, (n_bins, k))
    mask = rng.random((M, N)) < 0.6
    rows, cols = np.nonzero(mask)
    ptr = np.concatenate([[0], np.cumsum(mask.sum(1))]).astype(np.int64)
    bins = rng.integers(0, n_bins, size=rows.size).astype(np.int32)
    val = (Us[rows] * Vs[cols] * Ts[bins]).sum(1) * 10.0
    t = oracle.TensorTrajectory(M, N, n_bins, ptr, cols.astype(np.int32), bins, val,
                                rng.normal(0, 0.5, (M, k)), rng.normal(0, 0.5, (N, k)),
                                rng.normal(1, 0.1, (n_bins, k)), 1e-10)
    for _ in range(300):
        t.sweep()
    assert t.rmse() / val.std() < 1e-4


def test_t6_unit_time_factors_give_the_training_sse():
    _, ptr, col, bins, val, U, V, T = tensor_case(67)
    got = oracle.tensor_sse(ptr, col, bins, val, U, V, np.ones_like(T))
    assert got == pytest.approx(oracle.sse(ptr, col, val, U, V), rel=1e-13)


def test_time_bins_recipe():
    r = workload.make_config(1)
    b = workload.time_bins(r.row_ptr, workload.N_TIME_BINS, workload.time_seed(1))
    assert b.shape == (r.nnz,) and b.dtype == np.int32
    assert b.min() >= 0 and b.max() < workload.N_TIME_BINS
    again = workload.time_bins(r.row_ptr, workload.N_TIME_BINS, workload.time_seed(1))
    assert np.array_equal(b, again)
    # a user's ratings lie at or after its start: the spread within a user is bounded by
    # the exponential tail, far below the number of bins
    first = b[r.row_ptr[:-1]]
    assert np.median(np.abs(b - np.repeat(first, np.diff(r.row_ptr)))) < 1000
