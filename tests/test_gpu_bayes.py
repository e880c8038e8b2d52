"""Bayesian (BPMF / BPTF) Gibbs step on the GPU against the fp64 oracle, with the same
variates on both sides.

Bars:
- row draws: relative row error <= 1e-4, the half-sweep's own bar. The draw is the ALS
  system with Lambda / alpha in place of lambda n_s I plus one more right-hand-side term,
  solved by the same fp32 factorisation. Flagged rows must match and keep their value.
- hyperparameter draws: both sides are fp64. They differ only in summation order and in
  the factorisation variants, far below 1e-9 relative (Frobenius) for the well-conditioned
  posteriors here.
"""
import sys

import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROW_TOL = 1e-4
HYPER_TOL = 1e-9


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a, dtype=np.float32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).to("cuda:0")


def rel_rows(x, ref):
    return np.linalg.norm(x - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)


def spd(rng, D, scale=1.0):
    A = rng.normal(size=(D, D))
    return scale * (A @ A.T / D + np.eye(D))


def bartlett_variates(rng, D, nu_s):
    return (rng.chisquare(nu_s - np.arange(D)), rng.normal(size=D * (D - 1) // 2),
            rng.normal(size=D))


def small_matrix(M, N, seed, zero_users=3):
    """Prescribed user degrees with a few users and (by construction) some items without
    ratings; 8-16 ratings per user otherwise."""
    rng = np.random.default_rng(seed)
    deg = rng.integers(8, 17, size=M)
    deg[rng.choice(M, zero_users, replace=False)] = 0
    w = np.ones(N)
    w[:4] = 0.0  # items 0..3 are never sampled: rows without ratings on the item side
    return workload.make_custom(M, N, deg, seed, item_weights=w)


def check_gibbs_both_sides(M, N, ptr, col, val, D, alpha, seed, tuning=None, label=""):
    from paper_1108_2580_amd import ALS

    rng = np.random.default_rng(seed)
    U0 = (rng.normal(0, 0.3, size=(M, D))).astype(np.float32)
    V0 = (rng.normal(0, 0.3, size=(N, D))).astype(np.float32)
    csr = (ptr, col, val.astype(np.float64))
    csc = oracle.transpose(ptr, col, val, N)
    with ALS(M, N, ptr, col, val, D, tuning=tuning) as als:
        for side, fixed, prev, (p, i, v), n in (("users", V0, U0, csr, M),
                                                ("items", U0, V0, csc, N)):
            Lam = spd(rng, D, 0.5)
            mu = rng.normal(0, 0.2, size=D)
            z = rng.standard_normal((n, D), dtype=np.float32)
            log(f"  {label} gibbs side={side} D={D} alpha={alpha}")
            out = dev(prev)
            als.gibbs_half_sweep(side, dev(fixed), alpha, dev(Lam, np.float64),
                                 dev(mu, np.float64), dev(z), out, allow_flagged=True)
            xg = out.cpu().numpy()
            nfl = als.flagged_rows()
            xo, fl = oracle.gibbs_rows(p, i, v, fixed, alpha, Lam, mu, z, prev)
            assert nfl == int(fl.sum())
            ok = fl == 0
            r = rel_rows(xg[ok], xo[ok])
            log(f"    rows {ok.sum()} max rel {r.max():.2e} p99 {np.percentile(r, 99):.2e}")
            assert r.max() <= ROW_TOL
            assert np.array_equal(xg[~ok], prev[~ok])


@pytest.mark.parametrize("D", [1, 7, 10, 16, 17, 20, 33, 48, 64, 100, 128])
def test_gibbs_rows_match_oracle(D):
    M, N = 400, 260
    ptr, col, val = small_matrix(M, N, 300 + D)
    check_gibbs_both_sides(M, N, ptr, col, val, D, alpha=0.7, seed=D, label="small")


@pytest.mark.parametrize("D", [10, 20, 33, 100])
def test_gibbs_split_rows_and_batches(D):
    """Rows above the hub threshold are cut into chunks; a small workspace forces several
    batches."""
    M, N = 300, 900
    rng = np.random.default_rng(D)
    deg = rng.integers(5, 30, size=M)
    deg[:6] = [700, 520, 300, 260, 200, 130]
    ptr, col, val = workload.make_custom(M, N, deg, 77 + D)
    tun = dict(hub_threshold=64, chunk=48, workspace_bytes=40 * 1024 * (D // 4 + 4))
    check_gibbs_both_sides(M, N, ptr, col, val, D, alpha=1.3, seed=50 + D, tuning=tun,
                           label="split")


def test_gibbs_zero_noise_isotropic_prior_is_unweighted_ridge():
    """z = 0, mu = 0, Lambda = kappa I: the draw is the ridge solution with kappa / alpha."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(1)
    D = r.D
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    kappa, alpha = 3.0, 0.5
    log("gibbs z=0 isotropic")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        out = dev(U0)
        als.gibbs_half_sweep("users", dev(V0), alpha, dev(kappa * np.eye(D), np.float64),
                             dev(np.zeros(D), np.float64), dev(np.zeros((r.M, D))), out)
        xg = out.cpu().numpy()
    Fs = V0.astype(np.float64)
    for s in range(0, r.M, 97):
        a, b = r.row_ptr[s], r.row_ptr[s + 1]
        A = np.vstack([Fs[r.col[a:b]], np.sqrt(kappa / alpha) * np.eye(D)])
        y = np.concatenate([r.val[a:b].astype(np.float64), np.zeros(D)])
        want = np.linalg.lstsq(A, y, rcond=None)[0]
        assert np.linalg.norm(xg[s] - want) <= ROW_TOL * np.linalg.norm(want)


def test_gibbs_non_spd_prior_flags_rows_without_ratings():
    from paper_1108_2580_amd import ALS

    M, N, D = 60, 50, 6
    ptr, col, val = small_matrix(M, N, 5, zero_users=5)
    rng = np.random.default_rng(1)
    U0 = rng.normal(size=(M, D)).astype(np.float32)
    V0 = rng.normal(size=(N, D)).astype(np.float32)
    z = rng.standard_normal((M, D), dtype=np.float32)
    Lam = np.zeros((D, D))
    mu = np.zeros(D)
    log("gibbs non-SPD prior")
    with ALS(M, N, ptr, col, val, D) as als:
        out = dev(U0)
        als.gibbs_half_sweep("users", dev(V0), 1.0, dev(Lam, np.float64), dev(mu, np.float64),
                             dev(z), out, allow_flagged=True)
        xg = out.cpu().numpy()
        nfl = als.flagged_rows()
    xo, fl = oracle.gibbs_rows(ptr, col, val.astype(np.float64), V0, 1.0, Lam, mu, z, U0)
    assert nfl == int(fl.sum()) >= 5
    assert np.array_equal(xg[fl == 1], U0[fl == 1])
    ok = fl == 0
    assert rel_rows(xg[ok], xo[ok]).max() <= ROW_TOL


def test_gibbs_argument_errors():
    from paper_1108_2580_amd import ALS, ALSError, ALS_ERR_INVALID_ARG

    M, N, D = 30, 20, 4
    ptr, col, val = small_matrix(M, N, 9, zero_users=0)
    U = dev(np.zeros((M, D)))
    V = dev(np.zeros((N, D)))
    L = dev(np.eye(D), np.float64)
    m = dev(np.zeros(D), np.float64)
    z = dev(np.zeros((M, D)))
    log("gibbs argument errors")
    with ALS(M, N, ptr, col, val, D) as als:
        for a in (0.0, -1.0, float("inf")):
            with pytest.raises(ALSError) as e:
                als.gibbs_half_sweep("users", V, a, L, m, z, U)
            assert e.value.status == ALS_ERR_INVALID_ARG
        with pytest.raises(ALSError):
            als.gibbs_half_sweep("users", V, 1.0, L, m, U, U)  # z overlaps out
        als.set_weights(np.ones(col.size))
        with pytest.raises(ALSError):
            als.gibbs_half_sweep("users", V, 1.0, L, m, z, U)
        als.set_weights(None)
        als.gibbs_half_sweep("users", V, 1.0, L, m, z, U)
        with pytest.raises(ALSError):  # no hyperprior set yet
            als.sample_hyper("users", U, dev(np.ones(D), np.float64),
                             dev(np.zeros(D * (D - 1) // 2), np.float64),
                             dev(np.zeros(D), np.float64))
        with pytest.raises(ALSError):
            als.set_nw_prior("users", np.zeros(D), 1.0, np.eye(D), D - 1.5)
        bad = np.eye(D)
        bad[0, 1] = 0.5
        with pytest.raises(ALSError):
            als.set_nw_prior("users", np.zeros(D), 1.0, bad, D + 1.0)


@pytest.mark.parametrize("D", [1, 2, 5, 20, 33, 100, 128])
def test_hyper_sample_matches_oracle(D):
    from paper_1108_2580_amd import ALS

    M, N = 3000, 1700
    ptr, col, val = small_matrix(M, N, 11 + D, zero_users=0)
    rng = np.random.default_rng(900 + D)
    log(f"hyper sample D={D}")
    with ALS(M, N, ptr, col, val, D) as als:
        for side, n in (("users", M), ("items", N)):
            X = rng.normal(0.2, 0.6, size=(n, D)).astype(np.float32)
            mu0 = rng.normal(0, 0.1, size=D)
            W0inv = spd(rng, D, 0.3)
            beta0, nu0 = 2.0, D + 3.0
            als.set_nw_prior(side, mu0, beta0, W0inv, nu0)
            chi2, offd, zmu = bartlett_variates(rng, D, nu0 + n)
            mu_g, Lam_g = als.sample_hyper(side, dev(X), dev(chi2, np.float64),
                                           dev(offd, np.float64), dev(zmu, np.float64),
                                           check=True)
            mu_g, Lam_g = mu_g.cpu().numpy(), Lam_g.cpu().numpy()
            post = oracle.nw_posterior(X, mu0, beta0, W0inv, nu0)
            mu_o, Lam_o = oracle.nw_sample(post[0], post[1], post[2], chi2, offd, zmu)
            eL = np.linalg.norm(Lam_g - Lam_o) / np.linalg.norm(Lam_o)
            em = np.linalg.norm(mu_g - mu_o) / max(np.linalg.norm(mu_o), 1e-30)
            log(f"  side={side} rel Lambda {eL:.2e} rel mu {em:.2e}")
            assert eL <= HYPER_TOL and em <= HYPER_TOL


def test_hyper_sample_non_spd_is_reported():
    from paper_1108_2580_amd import ALS, ALSError, ALS_ERR_NOT_SPD

    M, N, D = 40, 30, 3
    ptr, col, val = small_matrix(M, N, 2, zero_users=0)
    log("hyper sample non-SPD")
    with ALS(M, N, ptr, col, val, D) as als:
        als.set_nw_prior("items", np.zeros(D), 0.0, -1e6 * np.eye(D), D + 1.0)
        X = dev(np.random.default_rng(0).normal(size=(N, D)))
        with pytest.raises(ALSError) as e:
            als.sample_hyper("items", X, dev(np.ones(D), np.float64),
                             dev(np.zeros(3), np.float64), dev(np.zeros(D), np.float64),
                             check=True)
        assert e.value.status == ALS_ERR_NOT_SPD


@pytest.mark.parametrize("k,iters", [(1, 3), (2, 1)])
def test_gibbs_chain_teacher_forced(k, iters):
    """A BPMF chain on a config (items then users per iteration: hyperparameters of the
    side, then its rows), every step checked against the oracle fed the GPU's inputs."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    D = r.D
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(4242 + k)
    alpha = 1.0 / 25.0
    csr = (r.row_ptr, r.col, r.val.astype(np.float64))
    csc = oracle.transpose(r.row_ptr, r.col, r.val, r.N)
    log(f"gibbs chain {r.name} iterations {iters}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        for side in ("users", "items"):
            als.set_nw_prior(side, np.zeros(D), 2.0, np.eye(D), D + 1.0)
        U, V = dev(U0), dev(V0)
        for it in range(iters):
            for side, X, fixed, (p, i, v), n in (("items", V, U, csc, r.N),
                                                 ("users", U, V, csr, r.M)):
                Xh, Fh = X.cpu().numpy(), fixed.cpu().numpy()
                chi2, offd, zmu = bartlett_variates(rng, D, D + 1.0 + n)
                mu_g, Lam_g = als.sample_hyper(side, X, dev(chi2, np.float64),
                                               dev(offd, np.float64), dev(zmu, np.float64),
                                               check=True)
                post = oracle.nw_posterior(Xh, np.zeros(D), 2.0, np.eye(D), D + 1.0)
                mu_o, Lam_o = oracle.nw_sample(post[0], post[1], post[2], chi2, offd, zmu)
                Lh = Lam_g.cpu().numpy()
                eL = np.linalg.norm(Lh - Lam_o) / np.linalg.norm(Lam_o)
                assert eL <= HYPER_TOL
                z = rng.standard_normal((n, D), dtype=np.float32)
                rm = als.gibbs_half_sweep(side, fixed, alpha, Lam_g, mu_g, dev(z), X, rmse=True)
                xo, fl = oracle.gibbs_rows(p, i, v, Fh, alpha, Lh, mu_g.cpu().numpy(), z, Xh)
                assert not fl.any()
                rr = rel_rows(X.cpu().numpy(), xo)
                log(f"  iter {it + 1} {side}: rel Lambda {eL:.1e}, rows max rel {rr.max():.2e}, "
                    f"training RMSE {rm:.4f}")
                assert rr.max() <= ROW_TOL


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 4])
def test_full_size_gibbs_sampled_rows(k):
    """Full-size workload: one Gibbs half-sweep per side from the seeded factors, checked on
    sampled rows (largest, smallest and random) that the oracle draws one by one."""
    from paper_1108_2580_amd import ALS
    from tests.test_gpu_full import sample_rows

    r = workload.make_config(k)
    D = r.D
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(77 + k)
    alpha = 1.0 / 25.0
    Lam = spd(rng, D, 2.0)
    mu = rng.normal(0, 0.05, size=D)
    val = r.val.astype(np.float64)
    csc = oracle.transpose(r.row_ptr, r.col, val, r.N)
    log(f"full-size gibbs {r.name}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        for side, fixed, prev, (p, i, v), n in (("items", U0, V0, csc, r.N),
                                                ("users", V0, U0, (r.row_ptr, r.col, val), r.M)):
            z = rng.standard_normal((n, D), dtype=np.float32)
            out = dev(prev)
            als.gibbs_half_sweep(side, dev(fixed), alpha, dev(Lam, np.float64),
                                 dev(mu, np.float64), dev(z), out)
            assert als.flagged_rows() == 0
            xg = out.cpu().numpy()
            rows = sample_rows(p, 5 + k)
            sub_ptr = np.concatenate([[0], np.cumsum(p[rows + 1] - p[rows])]).astype(np.int64)
            sub_idx = np.concatenate([i[p[s]:p[s + 1]] for s in rows])
            sub_val = np.concatenate([v[p[s]:p[s + 1]] for s in rows])
            xo, fl = oracle.gibbs_rows(sub_ptr, sub_idx, sub_val, fixed, alpha, Lam, mu, z[rows],
                                       prev[rows])
            assert not fl.any()
            rr = rel_rows(xg[rows], xo)
            log(f"  side={side}: {rows.size} sampled rows, max rel {rr.max():.2e}")
            assert rr.max() <= ROW_TOL
            assert np.isfinite(xg).all()
