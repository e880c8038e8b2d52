"""Pins of the oracle's BPTF pieces (tensor-model row draws, the time factors' Markov
chain, its Normal-Wishart posterior, and the rating precision) against facts that do not
come from the oracle:

- the full conditional of one bin, taken from the joint Gaussian of the whole chain, which
  the test assembles block by block from the chain's quadratic form (numpy solves);
- conjugacy, checked by density ratios with scipy's Wishart, normal and gamma densities:
  prior times likelihood over posterior must not depend on the parameter value;
- reductions to pinned pieces: unit time factors give the matrix model's row draw, and a
  chain of one bin is a plain Normal-Wishart sample of one row.

The model: r ~ N(sum_d U_ud V_id T_td, 1 / alpha); T_0 ~ N(mu_T, Lambda_T^{-1}) and
T_k ~ N(T_{k-1}, Lambda_T^{-1}); (mu_T, Lambda_T) Normal-Wishart; alpha ~ W(w0, nu0) in one
dimension (w0 times a chi-square with nu0 degrees of freedom).
"""
import numpy as np
import pytest

import oracle

scipy_stats = pytest.importorskip("scipy.stats")


def spd(rng, D, scale=1.0):
    A = rng.normal(size=(D, D))
    return scale * (A @ A.T / D + np.eye(D))


def chain_problem(rng, K, D, M=7, N=6, per_bin=(0, 6)):
    """Ratings grouped by time bin: ptr over bins, user and item indices, values."""
    counts = rng.integers(per_bin[0], per_bin[1] + 1, size=K)
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    n = int(ptr[-1])
    users = rng.integers(0, M, size=n).astype(np.int32)
    items = rng.integers(0, N, size=n).astype(np.int32)
    val = rng.integers(0, 101, size=n).astype(np.float64) / 20.0
    U = rng.normal(0, 0.6, size=(M, D))
    V = rng.normal(0, 0.6, size=(N, D))
    return ptr, users, items, val, U, V


def joint_chain(ptr, users, items, val, U, V, alpha, Lam, mu):
    """Precision P (K D x K D) and linear term h of the joint Gaussian of all bins, from
    -1/2 (T_0 - mu)' Lam (T_0 - mu) - 1/2 sum_k (T_k - T_{k-1})' Lam (T_k - T_{k-1})
    - alpha / 2 sum (r - f . T_k)^2, expanded block by block."""
    K, D = ptr.size - 1, U.shape[1]
    P = np.zeros((K * D, K * D))
    h = np.zeros(K * D)
    blk = lambda i: slice(i * D, (i + 1) * D)
    P[blk(0), blk(0)] += Lam
    h[blk(0)] += Lam @ mu
    for k in range(1, K):
        P[blk(k), blk(k)] += Lam
        P[blk(k - 1), blk(k - 1)] += Lam
        P[blk(k), blk(k - 1)] -= Lam
        P[blk(k - 1), blk(k)] -= Lam
    for k in range(K):
        for q in range(ptr[k], ptr[k + 1]):
            f = U[users[q]] * V[items[q]]
            P[blk(k), blk(k)] += alpha * np.outer(f, f)
            h[blk(k)] += alpha * val[q] * f
    return P, h


def conditional_draw(P, h, T, k, z):
    """Bin k given the other bins: precision P_kk, mean P_kk^{-1} (h_k - sum_j P_kj T_j),
    then mean + chol(P_kk)^{-T} z."""
    D = T.shape[1]
    K = T.shape[0]
    rows = slice(k * D, (k + 1) * D)
    Pkk = P[rows, rows]
    rest = h[rows].copy()
    for j in range(K):
        if j != k:
            rest -= P[rows, j * D:(j + 1) * D] @ T[j]
    mean = np.linalg.solve(Pkk, rest)
    L = np.linalg.cholesky(Pkk)
    return mean + np.linalg.solve(L.T, z)


# ---- rows under the tensor model ---------------------------------------------------------------

@pytest.mark.parametrize("D", [1, 4])
def test_bt1_unit_time_factors_give_the_matrix_draw(D):
    rng = np.random.default_rng(70 + D)
    M, N = 9, 8
    counts = rng.integers(0, 6, size=M)
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    n = int(ptr[-1])
    idx = rng.integers(0, N, size=n).astype(np.int32)
    bins = rng.integers(0, 3, size=n).astype(np.int32)
    val = rng.integers(0, 101, size=n).astype(np.float64)
    F = rng.normal(0, 0.5, size=(N, D))
    Lam, mu = spd(rng, D, 1.5), rng.normal(0, 0.3, size=D)
    z = rng.normal(size=(M, D))
    X0 = rng.normal(size=(M, D))
    xt, ft = oracle.tensor_gibbs_rows(ptr, idx, bins, val, F, np.ones((3, D)), 0.7, Lam, mu, z, X0)
    xm, fm = oracle.gibbs_rows(ptr, idx, val, F, 0.7, Lam, mu, z, X0)
    assert not ft.any() and not fm.any()
    np.testing.assert_allclose(xt, xm, rtol=1e-13, atol=1e-13)


def test_bt2_tensor_row_uses_the_elementwise_product():
    """A tensor row draw equals the matrix draw over explicitly formed product vectors."""
    rng = np.random.default_rng(72)
    D, n = 3, 7
    F1, F2 = rng.normal(size=(5, D)), rng.normal(size=(4, D))
    i1 = rng.integers(0, 5, size=n).astype(np.int32)
    i2 = rng.integers(0, 4, size=n).astype(np.int32)
    val = rng.normal(size=n)
    ptr = np.array([0, n], dtype=np.int64)
    Lam, mu, z = spd(rng, D), rng.normal(size=D), rng.normal(size=(1, D))
    xt, _ = oracle.tensor_gibbs_rows(ptr, i1, i2, val, F1, F2, 1.3, Lam, mu, z, np.zeros((1, D)))
    Fs = F1[i1] * F2[i2]
    xm, _ = oracle.gibbs_rows(ptr, np.arange(n, dtype=np.int32), val, Fs, 1.3, Lam, mu, z,
                              np.zeros((1, D)))
    np.testing.assert_allclose(xt, xm, rtol=1e-12, atol=1e-12)


# ---- the time chain --------------------------------------------------------------------------

@pytest.mark.parametrize("K,D", [(1, 2), (2, 3), (5, 3), (8, 2)])
def test_bt3_bins_are_the_joint_gaussians_conditionals(K, D):
    rng = np.random.default_rng(80 + 10 * K + D)
    ptr, users, items, val, U, V = chain_problem(rng, K, D)
    if K > 2:
        ptr[2:] -= ptr[2] - ptr[1]  # bin 1 has no ratings
        users, items, val = users[:ptr[-1]], items[:ptr[-1]], val[:ptr[-1]]
    alpha = 1.7
    Lam, mu = spd(rng, D, 2.0), rng.normal(0, 0.4, size=D)
    T0 = rng.normal(0, 0.5, size=(K, D))
    z = rng.normal(size=(K, D))
    P, h = joint_chain(ptr, users, items, val, U, V, alpha, Lam, mu)
    T = T0.copy()
    for parity in (0, 1):
        Tn, fl = oracle.time_rows(ptr, users, items, val, U, V, alpha, Lam, mu, z, parity, T)
        assert not fl.any()
        for k in range(K):
            if k % 2 == parity:
                want = conditional_draw(P, h, T, k, z[k])
                np.testing.assert_allclose(Tn[k], want, rtol=1e-10, atol=1e-11)
            else:
                assert np.array_equal(Tn[k], T[k])
        T = Tn


def test_bt4_single_bin_chain_is_the_matrix_prior_draw():
    """One bin: the chain prior is N(mu_T, Lambda_T^{-1}) alone, so the draw is the row
    draw of the tensor model with that prior."""
    rng = np.random.default_rng(90)
    D = 3
    ptr, users, items, val, U, V = chain_problem(rng, 1, D, per_bin=(4, 6))
    Lam, mu, z = spd(rng, D), rng.normal(size=D), rng.normal(size=(1, D))
    Tt, _ = oracle.time_rows(ptr, users, items, val, U, V, 0.9, Lam, mu, z, 0, np.zeros((1, D)))
    Tg, _ = oracle.tensor_gibbs_rows(ptr, users, items, val, U, V, 0.9, Lam, mu, z,
                                     np.zeros((1, D)))
    np.testing.assert_allclose(Tt, Tg, rtol=1e-13, atol=1e-13)


def test_bt5_empty_interior_bin_without_noise_is_the_neighbours_mean():
    rng = np.random.default_rng(91)
    D, K = 2, 4
    ptr = np.array([0, 3, 3, 5, 6], dtype=np.int64)  # bin 1 empty
    users = rng.integers(0, 5, size=6).astype(np.int32)
    items = rng.integers(0, 5, size=6).astype(np.int32)
    val = rng.normal(size=6)
    U, V = rng.normal(size=(5, D)), rng.normal(size=(5, D))
    T0 = rng.normal(size=(K, D))
    Tn, _ = oracle.time_rows(ptr, users, items, val, U, V, 1.0, spd(rng, D), np.zeros(D),
                             np.zeros((K, D)), 1, T0)
    np.testing.assert_allclose(Tn[1], 0.5 * (T0[0] + T0[2]), rtol=1e-13, atol=1e-14)


# ---- conjugate posteriors (density ratios) -----------------------------------------------------

def nw_logpdf(mu, Lam, mu0, beta0, W, nu):
    st = scipy_stats
    return (st.wishart.logpdf(Lam, df=nu, scale=W)
            + st.multivariate_normal.logpdf(mu, mean=mu0, cov=np.linalg.inv(beta0 * Lam)))


@pytest.mark.parametrize("K,D", [(1, 2), (4, 2), (9, 3)])
def test_bt6_time_posterior_is_conjugate(K, D):
    st = scipy_stats
    rng = np.random.default_rng(100 + K + D)
    T = np.cumsum(rng.normal(0, 0.4, size=(K, D)), axis=0) + rng.normal(size=D)
    mu0, beta0, nu0 = rng.normal(size=D), 1.5, D + 1.5
    W0 = spd(rng, D, 0.8)
    mu_s, beta_s, Winv_s, nu_s = oracle.time_posterior(T, mu0, beta0, np.linalg.inv(W0), nu0)
    W_s = np.linalg.inv(Winv_s)
    logs = []
    for _ in range(6):
        Lam = st.wishart.rvs(df=D + 3, scale=np.eye(D) / D, random_state=rng)
        Lam = np.atleast_2d(Lam)
        mu = rng.normal(size=D)
        cov = np.linalg.inv(Lam)
        lik = st.multivariate_normal.logpdf(T[0], mean=mu, cov=cov)
        for k in range(1, K):
            lik += st.multivariate_normal.logpdf(T[k] - T[k - 1], mean=np.zeros(D), cov=cov)
        logs.append(nw_logpdf(mu, Lam, mu0, beta0, W0, nu0) + lik
                    - nw_logpdf(mu, Lam, mu_s, beta_s, W_s, nu_s))
    logs = np.array(logs)
    assert np.ptp(logs) <= 1e-8 * max(1.0, np.abs(logs).max())


def test_bt7_one_bin_posterior_is_the_one_row_posterior():
    rng = np.random.default_rng(110)
    D = 3
    T = rng.normal(size=(1, D))
    mu0, W0inv = rng.normal(size=D), spd(rng, D)
    a = oracle.time_posterior(T, mu0, 2.0, W0inv, D + 2.0)
    b = oracle.nw_posterior(T, mu0, 2.0, W0inv, D + 2.0)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-14, atol=1e-14)


def test_bt8_alpha_posterior_is_conjugate():
    st = scipy_stats
    rng = np.random.default_rng(120)
    n = 57
    resid = rng.normal(0, 2.0, size=n)
    sse = float(resid @ resid)
    w0, nu0 = 0.3, 4.0
    w_s, nu_s = oracle.alpha_posterior(sse, n, w0, nu0)
    logs = []
    for alpha in (0.05, 0.2, 0.9, 3.0):
        prior = st.gamma.logpdf(alpha, a=nu0 / 2, scale=2 * w0)
        lik = st.norm.logpdf(resid, scale=1 / np.sqrt(alpha)).sum()
        logs.append(prior + lik - st.gamma.logpdf(alpha, a=nu_s / 2, scale=2 * w_s))
    assert np.ptp(logs) <= 1e-9 * max(1.0, np.abs(logs).max())
