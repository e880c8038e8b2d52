"""Pins of the oracle's weighted ALS (wALS) against facts that do not come from it.

The paper lists weighted ALS beside ALS (Sec. 2 and Sec. 4) without defining its
weighting. The reading used here: every stored rating carries a non-negative
weight c, and a row minimises sum_j c_j (r_j - f_j . x)^2 + lambda n_s ||x||^2 (the
regulariser keeps the count n_s, so unit weights are plain ALS). Each test fixes a
property that this definition or plain mathematics determines.
"""
import numpy as np
import pytest

import oracle
from tests.test_oracle_pins import np_transpose, rand_csr


def rand_weights(rng, n, lo=0.25, hi=4.0):
    return np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))


def test_w1_unit_weights_are_plain_als():
    rng = np.random.default_rng(101)
    M, N, D, lam = 40, 30, 6, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    F = rng.normal(0, 0.2, size=(N, D))
    X0 = rng.normal(size=(M, D))
    a, fa = oracle.half_sweep(ptr, idx, val, F, lam, X0)
    b, fb = oracle.half_sweep(ptr, idx, val, F, lam, X0, w=np.ones(val.size))
    assert np.array_equal(a, b) and np.array_equal(fa, fb)


@pytest.mark.parametrize("D", [1, 3, 6])
def test_w2_matches_weighted_lstsq(D):
    # textbook weighted ridge: scale each equation by sqrt(c) and stack sqrt(lambda n) I
    rng = np.random.default_rng(102 + D)
    M, N, lam = 15, 30, 0.37
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    w = rand_weights(rng, val.size)
    F = rng.normal(0, 0.7, size=(N, D))
    X, fl = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)), w=w)
    assert (fl == 0).all()
    for s in range(M):
        sl = slice(ptr[s], ptr[s + 1])
        js, r, c = idx[sl], val[sl], w[sl]
        n = js.size
        Aaug = np.vstack([np.sqrt(c)[:, None] * F[js], np.sqrt(lam * n) * np.eye(D)])
        baug = np.concatenate([np.sqrt(c) * r, np.zeros(D)])
        x_ls = np.linalg.lstsq(Aaug, baug, rcond=None)[0]
        np.testing.assert_allclose(X[s], x_ls, rtol=1e-10, atol=1e-12)


def test_w3_weighted_gradient_zero():
    rng = np.random.default_rng(103)
    M, N, D, lam = 40, 25, 6, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.4, min_deg=1)
    w = rand_weights(rng, val.size)
    F = rng.normal(0, 0.1, size=(N, D))
    X, _ = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)), w=w)
    for s in range(M):
        sl = slice(ptr[s], ptr[s + 1])
        js, r, c = idx[sl], val[sl], w[sl]
        # gradient of sum c (r - f.x)^2 + lam n |x|^2, straight from the ratings
        resid = F[js] @ X[s] - r
        grad = 2.0 * (F[js].T @ (c * resid) + lam * js.size * X[s])
        assert np.linalg.norm(grad) <= 1e-9 * (np.linalg.norm(F[js].T @ (c * r)) + 1.0)


def test_w4_weighted_objective_monotone():
    rng = np.random.default_rng(104)
    M, N, D, lam = 60, 45, 5, 0.05
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=2)
    w = rand_weights(rng, val.size)
    t = oracle.Trajectory(M, N, ptr, idx, val, rng.normal(0, 0.1, size=(M, D)),
                          rng.normal(0, 0.1, size=(N, D)), lam, w=w)
    L = [t.objective()]
    for _ in range(6):
        t.step("items")
        L.append(t.objective())
        t.step("users")
        L.append(t.objective())
    for a, b in zip(L, L[1:]):
        assert b <= a * (1 + 1e-12)
    assert L[-1] < 0.5 * L[0]


def test_w5_integer_weight_is_repeated_rating():
    # a weight k puts the same terms into G and b as k stored copies of the rating
    rng = np.random.default_rng(105)
    N, D, lam = 20, 5, 0.2
    js = rng.choice(N, size=7, replace=False).astype(np.int32)
    r = rng.integers(0, 101, size=7).astype(np.float64)
    k = rng.integers(1, 5, size=7)
    F = rng.normal(size=(N, D))
    A_w, b_w = oracle.normal_equations(0, np.array([0, 7]), js, r, F, lam, w=k.astype(np.float64))
    jr, rr = np.repeat(js, k), np.repeat(r, k)
    A_r, b_r = oracle.normal_equations(0, np.array([0, jr.size]), jr, rr, F, lam)
    # same Gram and right-hand side; the regulariser counts stored ratings (7 vs sum k)
    np.testing.assert_allclose(A_w - lam * 7 * np.eye(D), A_r - lam * jr.size * np.eye(D),
                               rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(b_w, b_r, rtol=1e-13, atol=1e-10)


def test_w6_zero_weight_drops_the_rating_but_not_its_count():
    rng = np.random.default_rng(106)
    N, D, lam = 20, 4, 0.3
    js = rng.choice(N, size=6, replace=False).astype(np.int32)
    r = rng.integers(0, 101, size=6).astype(np.float64)
    w = rand_weights(rng, 6)
    w[2] = 0.0
    F = rng.normal(size=(N, D))
    A_w, b_w = oracle.normal_equations(0, np.array([0, 6]), js, r, F, lam, w=w)
    keep = np.array([0, 1, 3, 4, 5])
    A_k, b_k = oracle.normal_equations(0, np.array([0, 5]), js[keep], r[keep], F, lam, w=w[keep])
    np.testing.assert_allclose(A_w, A_k + lam * np.eye(D), rtol=1e-14, atol=1e-13)
    np.testing.assert_allclose(b_w, b_k, rtol=1e-14, atol=1e-13)


def test_w7_single_rating_closed_form():
    # n = 1: (c f f^T + lam I) x = c r f  gives  x = c r f / (c |f|^2 + lam)
    rng = np.random.default_rng(107)
    D, lam = 6, 0.4
    F = rng.normal(size=(5, D))
    for j in range(5):
        r, c = float(rng.integers(0, 101)), float(rand_weights(rng, 1)[0])
        X, _ = oracle.half_sweep(np.array([0, 1]), np.array([j], dtype=np.int32), np.array([r]), F,
                                 lam, np.zeros((1, D)), w=np.array([c]))
        np.testing.assert_allclose(X[0], c * r * F[j] / (c * (F[j] @ F[j]) + lam), rtol=1e-12)


def test_w8_weights_travel_with_the_transpose():
    # the user half-sweep on (A, C) equals the item half-sweep on (A^T, C^T), the
    # transposed weights built independently by a numpy sort
    rng = np.random.default_rng(108)
    M, N, D, lam = 30, 20, 4, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.35, min_deg=1)
    w = rand_weights(rng, val.size)
    V = rng.normal(0, 0.1, size=(N, D))
    Xu, _ = oracle.half_sweep(ptr, idx, val, V, lam, np.zeros((M, D)), w=w)
    tptr, tidx, tval = np_transpose(ptr, idx, val, N)
    _, _, tw = np_transpose(ptr, idx, w, N)
    cptr, cidx, cval = oracle.transpose(tptr, tidx, tval, M)
    cw = oracle.transpose(tptr, tidx, tw, M)[2]
    Xi, _ = oracle.half_sweep(cptr, cidx, cval, V, lam, np.zeros((M, D)), w=cw)
    assert np.array_equal(Xu, Xi)
    # and the trajectory's own transposed weights agree with the independent ones
    t = oracle.Trajectory(M, N, ptr, idx, val, np.zeros((M, D)), V, lam, w=w)
    assert np.array_equal(t.w_t, tw)


def test_w9_weighted_sse():
    rng = np.random.default_rng(109)
    M, N, D = 20, 15, 3
    ptr, idx, val = rand_csr(rng, M, N, 0.4, min_deg=1)
    w = rand_weights(rng, val.size)
    U = rng.normal(size=(M, D))
    V = rng.normal(size=(N, D))
    rows = np.repeat(np.arange(M), np.diff(ptr))
    e = val - np.einsum("kd,kd->k", U[rows], V[idx])
    np.testing.assert_allclose(oracle.sse(ptr, idx, val, U, V, w=w), np.sum(w * e * e), rtol=1e-12)
    np.testing.assert_allclose(oracle.sse(ptr, idx, val, U, V), np.sum(e * e), rtol=1e-12)
