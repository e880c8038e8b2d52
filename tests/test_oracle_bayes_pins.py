"""Pins of the oracle's Bayesian (BPMF / BPTF) Gibbs step against facts that do not come
from the oracle: textbook ridge regression, the stationarity of the log posterior, the
covariance of the drawn noise (through numpy's own Cholesky factor), the conjugacy of the
Normal-Wishart update (batch equals sequential), the flat-prior limit (numpy's sample
covariance), the inverse relation of the Wishart scale, and the Wishart moments.

The model: r ~ N(u . v, 1 / alpha); each row has the prior N(mu, Lambda^{-1}); (mu, Lambda)
has a Normal-Wishart hyperprior. A row's conditional is Gaussian with precision
Lambda* = Lambda + alpha sum f f^T and mean mu* = Lambda*^{-1} (alpha sum r f + Lambda mu).
"""
import numpy as np
import pytest

import oracle
from tests.test_oracle_pins import rand_csr


def spd(rng, D, scale=1.0):
    A = rng.normal(size=(D, D))
    return scale * (A @ A.T / D + np.eye(D))


def one_row(rng, D, n, scale=0.5):
    F = rng.normal(0, scale, size=(n + 3, D))
    idx = rng.choice(n + 3, size=n, replace=False).astype(np.int32)
    val = rng.integers(0, 101, size=n).astype(np.float64)
    ptr = np.array([0, n], dtype=np.int64)
    return ptr, np.sort(idx), val, F


# ---- row conditional ------------------------------------------------------------------------

@pytest.mark.parametrize("D", [1, 3, 6])
def test_b1_zero_noise_isotropic_prior_is_ridge(D):
    rng = np.random.default_rng(40 + D)
    ptr, idx, val, F = one_row(rng, D, 9)
    alpha, kappa = 2.5, 0.7
    x, fl = oracle.gibbs_rows(ptr, idx, val, F, alpha, kappa * np.eye(D), np.zeros(D),
                              np.zeros((1, D)), np.zeros((1, D)))
    assert fl[0] == 0
    Fs = F[idx]
    A = np.vstack([Fs, np.sqrt(kappa / alpha) * np.eye(D)])
    y = np.concatenate([val, np.zeros(D)])
    want = np.linalg.lstsq(A, y, rcond=None)[0]
    np.testing.assert_allclose(x[0], want, rtol=1e-11, atol=1e-12)


def test_b2_zero_noise_is_the_posterior_mode():
    """With z = 0 the draw is the conditional mean, where the gradient of the log posterior
    alpha sum (r - x.f) f - Lambda (x - mu) vanishes (computed from the ratings)."""
    rng = np.random.default_rng(41)
    M, N, D = 25, 30, 5
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    F = rng.normal(0, 0.4, size=(N, D))
    Lam = spd(rng, D, 2.0)
    mu = rng.normal(0, 0.3, size=D)
    alpha = 0.8
    X, fl = oracle.gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, np.zeros((M, D)),
                              np.zeros((M, D)))
    assert not fl.any()
    for s in range(M):
        f = F[idx[ptr[s]:ptr[s + 1]]]
        r = val[ptr[s]:ptr[s + 1]]
        g = alpha * f.T @ (r - f @ X[s]) - Lam @ (X[s] - mu)
        scale = alpha * np.abs(f.T @ r).sum() + np.abs(Lam @ mu).sum() + 1
        assert np.linalg.norm(g) <= 1e-11 * scale


def test_b3_noise_has_the_conditional_covariance():
    """x(z) - x(0) = L*^{-T} z, i.e. Lambda* (x(z) - x(0)) = L* z, with L* numpy's own
    Cholesky factor of Lambda* = Lambda + alpha sum f f^T (built here from the ratings); so
    the noise has covariance Lambda*^{-1}. Linear in z."""
    rng = np.random.default_rng(42)
    M, N, D = 20, 25, 6
    ptr, idx, val = rand_csr(rng, M, N, 0.35, min_deg=1)
    F = rng.normal(0, 0.5, size=(N, D))
    Lam = spd(rng, D)
    mu = rng.normal(size=D)
    alpha = 1.7
    z1 = rng.normal(size=(M, D))
    z2 = rng.normal(size=(M, D))
    prev = np.zeros((M, D))
    x0, _ = oracle.gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, np.zeros((M, D)), prev)
    x1, _ = oracle.gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, z1, prev)
    x12, _ = oracle.gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, z1 + z2, prev)
    x2, _ = oracle.gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, z2, prev)
    for s in range(M):
        f = F[idx[ptr[s]:ptr[s + 1]]]
        Ls = Lam + alpha * f.T @ f
        L = np.linalg.cholesky(Ls)
        np.testing.assert_allclose(Ls @ (x1[s] - x0[s]), L @ z1[s], rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(x12 - x0, (x1 - x0) + (x2 - x0), rtol=1e-9, atol=1e-11)


def test_b4_row_without_ratings_is_a_prior_draw():
    rng = np.random.default_rng(43)
    D = 4
    ptr = np.array([0, 0, 2], dtype=np.int64)
    idx = np.array([0, 1], dtype=np.int32)
    val = np.array([3.0, 4.0])
    F = rng.normal(size=(2, D))
    Lam = spd(rng, D)
    mu = rng.normal(size=D)
    z = rng.normal(size=(2, D))
    X, fl = oracle.gibbs_rows(ptr, idx, val, F, 1.3, Lam, mu, z, np.zeros((2, D)))
    assert not fl.any()
    np.testing.assert_allclose(Lam @ (X[0] - mu), np.linalg.cholesky(Lam) @ z[0], rtol=1e-11,
                               atol=1e-12)


def test_b5_non_spd_prior_is_flagged_and_row_kept():
    D = 3
    ptr = np.array([0, 0], dtype=np.int64)
    prev = np.full((1, D), 7.0)
    X, fl = oracle.gibbs_rows(ptr, np.zeros(0, np.int32), np.zeros(0), np.ones((1, D)), 1.0,
                              np.zeros((D, D)), np.zeros(D), np.ones((1, D)), prev)
    assert fl[0] == 1 and np.array_equal(X, prev)


# ---- Normal-Wishart posterior ------------------------------------------------------------------

def test_b6_conjugate_update_batch_equals_sequential():
    rng = np.random.default_rng(44)
    D = 4
    X = rng.normal(0.3, 0.8, size=(37, D))
    mu0 = rng.normal(size=D)
    W0inv = spd(rng, D, 0.5)
    beta0, nu0 = 2.0, D + 1.0
    batch = oracle.nw_posterior(X, mu0, beta0, W0inv, nu0)
    m1, b1, Wi1, v1 = oracle.nw_posterior(X[:15], mu0, beta0, W0inv, nu0)
    seq = oracle.nw_posterior(X[15:], m1, b1, Wi1, v1)
    np.testing.assert_allclose(batch[0], seq[0], rtol=1e-12, atol=1e-13)
    assert batch[1] == seq[1] and batch[3] == seq[3]
    np.testing.assert_allclose(batch[2], seq[2], rtol=1e-12)


def test_b7_flat_prior_gives_the_sample_scatter():
    rng = np.random.default_rng(45)
    D = 5
    X = rng.normal(1.0, 2.0, size=(60, D))
    mu_s, beta_s, Winv, nu_s = oracle.nw_posterior(X, np.zeros(D), 0.0, np.zeros((D, D)), D)
    np.testing.assert_allclose(mu_s, X.mean(axis=0), rtol=1e-13)
    np.testing.assert_allclose(Winv, (X.shape[0] - 1) * np.cov(X.T), rtol=1e-12)
    assert beta_s == 60.0 and nu_s == 60.0 + D


# ---- Normal-Wishart draw -----------------------------------------------------------------------

def test_b8_unit_variates_give_the_scale_matrix():
    """chi2 = 1, off-diagonal normals 0, mu normals 0: Lambda = W* (the inverse of the given
    W*^{-1}) and mu = mu*."""
    rng = np.random.default_rng(46)
    D = 5
    Winv = spd(rng, D, 3.0)
    mu_s = rng.normal(size=D)
    mu, Lam = oracle.nw_sample(mu_s, 4.0, Winv, np.ones(D), np.zeros(D * (D - 1) // 2),
                               np.zeros(D))
    np.testing.assert_allclose(Lam @ Winv, np.eye(D), atol=1e-12)
    assert np.array_equal(mu, mu_s)


def test_b9_mean_draw_has_covariance_of_beta_lambda_inverse():
    """mu - mu* = R^{-T} zmu with R numpy's Cholesky factor of beta* Lambda."""
    rng = np.random.default_rng(47)
    D = 4
    Winv = spd(rng, D)
    mu_s = rng.normal(size=D)
    chi2 = rng.chisquare(20.0 - np.arange(D))
    offd = rng.normal(size=D * (D - 1) // 2)
    zmu = rng.normal(size=D)
    mu, Lam = oracle.nw_sample(mu_s, 3.0, Winv, chi2, offd, zmu)
    R = np.linalg.cholesky(3.0 * Lam)
    np.testing.assert_allclose(3.0 * Lam @ (mu - mu_s), R @ zmu, rtol=1e-10, atol=1e-12)


def test_b10_wishart_moments():
    """Over many draws with numpy's chi-square and normal variates: E[Lambda] = nu* W* and
    E[Lambda^{-1}] = W*^{-1} / (nu* - D - 1) (Wishart and inverse-Wishart means)."""
    rng = np.random.default_rng(48)
    D, nu, n = 3, 9.0, 20000
    Winv = spd(rng, D, 2.0)
    W = np.linalg.inv(Winv)
    acc = np.zeros((D, D))
    acc_inv = np.zeros((D, D))
    for _ in range(n):
        chi2 = rng.chisquare(nu - np.arange(D))
        offd = rng.normal(size=D * (D - 1) // 2)
        _, Lam = oracle.nw_sample(np.zeros(D), 1.0, Winv, chi2, offd, np.zeros(D))
        acc += Lam
        acc_inv += np.linalg.inv(Lam)
    mean = acc / n
    sd = np.sqrt(nu * (W ** 2 + np.outer(np.diag(W), np.diag(W))) / n)
    assert np.all(np.abs(mean - nu * W) <= 5 * sd)
    target = Winv / (nu - D - 1)
    assert np.linalg.norm(acc_inv / n - target) <= 0.05 * np.linalg.norm(target)
