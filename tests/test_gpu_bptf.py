"""BPTF's Gibbs step on the GPU (als_tensor_gibbs_half_sweep, als_sample_time_hyper,
als_tensor_sample_alpha) against the fp64 oracle, with the same variates on both sides.

Bars:
- row and time-bin draws: relative row error <= 1e-4, the half-sweep's own bar. A draw
  is the tensor ALS system with the prior image in place of lambda n_s I (scaled per bin
  for the chain) plus the prior's right-hand side, solved by the same fp32 factorisation.
- the chain's hyperparameter draw: fp64 on both sides, differing only in summation order
  and factorisation variants: 1e-9 relative (Frobenius).
- alpha: chi2 / (1 / w0 + sse), where the device's sse sums squares of fp32 three-way
  predictions in fp64. A prediction carries a relative rounding of about D 2^-24 of its
  terms' magnitudes, so sse, and with it alpha, agrees to 1e-5 relative at these sizes.
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
ALPHA_TOL = 1e-5


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


def problem(M, N, n_bins, D, seed, zero_users=2, deg=(6, 30), empty_bins=(3,), empty_last=True):
    """Ratings with a few users without ratings, the listed bins (and the last bin, with
    empty_last) without ratings, and seeded factors (T around 1)."""
    rng = np.random.default_rng(seed)
    degs = rng.integers(deg[0], deg[1], size=M)
    degs[rng.choice(M, zero_users, replace=False)] = 0
    ptr, col, val = workload.make_custom(M, N, degs, seed)
    last = n_bins - 1 if empty_last else n_bins
    allowed = np.array([b for b in range(last) if b not in empty_bins], dtype=np.int32)
    bins = allowed[rng.integers(0, allowed.size, size=col.size)]
    U = rng.normal(0, 0.5, size=(M, D)).astype(np.float32)
    V = rng.normal(0, 0.5, size=(N, D)).astype(np.float32)
    T = rng.normal(1.0, 0.2, size=(n_bins, D)).astype(np.float32)
    return ptr, col, val, bins, U, V, T


def groupings(M, N, n_bins, ptr, col, bins, val):
    t = oracle.TensorTrajectory(M, N, n_bins, ptr, col, bins, val.astype(np.float64),
                                np.zeros((M, 1)), np.zeros((N, 1)), np.zeros((n_bins, 1)), 0.0)
    return t.by_user, t.by_item, t.by_bin


@pytest.mark.parametrize("D", [1, 7, 16, 20, 33, 64, 100, 128])
def test_user_and_item_draws_match_oracle(D):
    from paper_1108_2580_amd import ALS

    M, N, K = 300, 200, 30
    ptr, col, val, bins, U, V, T = problem(M, N, K, D, 600 + D)
    by_user, by_item, _ = groupings(M, N, K, ptr, col, bins, val)
    rng = np.random.default_rng(610 + D)
    alpha = 0.05
    with ALS(M, N, ptr, col, val, D) as als:
        als.set_time_bins(K, bins)
        for mode, (p, i1, i2, v), F1, F2, X in (("items", by_item, U, T, V),
                                                ("users", by_user, V, T, U)):
            Lam, mu = spd(rng, D, 0.7), rng.normal(0, 0.2, size=D)
            z = rng.standard_normal((X.shape[0], D), dtype=np.float32)
            Ud, Vd, Td = dev(U), dev(V), dev(T)
            log(f"  bptf draw mode={mode} D={D}")
            als.tensor_gibbs_half_sweep(mode, Ud, Vd, Td, alpha, dev(Lam, np.float64),
                                        dev(mu, np.float64), dev(z), allow_flagged=True)
            xg = (Vd if mode == "items" else Ud).cpu().numpy()
            xo, fl = oracle.tensor_gibbs_rows(p, i1, i2, v, F1, F2, alpha, Lam, mu, z, X)
            assert als.flagged_rows() == int(fl.sum())
            ok = fl == 0
            r = rel_rows(xg[ok], xo[ok])
            log(f"    rows {ok.sum()} max rel {r.max():.2e}")
            assert r.max() <= ROW_TOL
            # the other factors are untouched
            assert np.array_equal(Td.cpu().numpy(), T)


def check_chain(M, N, K, D, seed, tuning=None, empty_bins=(3,), deg=(6, 30), empty_last=True,
                label=""):
    from paper_1108_2580_amd import ALS

    ptr, col, val, bins, U, V, T = problem(M, N, K, D, seed, deg=deg, empty_bins=empty_bins,
                                           empty_last=empty_last)
    _, _, (p, i1, i2, v) = groupings(M, N, K, ptr, col, bins, val)
    rng = np.random.default_rng(seed + 1)
    alpha = 0.05
    Lam, mu = spd(rng, D, 3.0), rng.normal(1.0, 0.1, size=D)
    z = rng.standard_normal((K, D), dtype=np.float32)
    with ALS(M, N, ptr, col, val, D, tuning=tuning) as als:
        als.set_time_bins(K, bins)
        Ud, Vd, Td = dev(U), dev(V), dev(T)
        log(f"  {label} chain D={D} K={K}")
        rm = als.tensor_gibbs_half_sweep("bins", Ud, Vd, Td, alpha, dev(Lam, np.float64),
                                         dev(mu, np.float64), dev(z), rmse=True)
        rm_in = als.rmse_in()
        tg = Td.cpu().numpy()
        assert als.flagged_rows() == 0
    # the entering state's RMSE covers every rating: the even pass's residuals plus the odd
    # pass's, both of the bins as they entered the chain
    by_user = groupings(M, N, K, ptr, col, bins, val)[0]
    ro_in = np.sqrt(oracle.tensor_sse(*by_user, U, V, T) / col.size)
    log(f"    entering rmse gpu {rm_in:.9f} oracle {ro_in:.9f}")
    assert abs(rm_in - ro_in) <= 1e-5
    # the oracle draws the even bins, then the odd bins given the new even ones
    to, fl0 = oracle.time_rows(p, i1, i2, v, U, V, alpha, Lam, mu, z, 0, T)
    # the odd pass reads the GPU's even bins, so each pass is checked from identical inputs
    te = T.astype(np.float64).copy()
    te[0::2] = tg[0::2]
    to1, fl1 = oracle.time_rows(p, i1, i2, v, U, V, alpha, Lam, mu, z, 1, te)
    assert not fl0.any() and not fl1.any()
    r_even = rel_rows(tg[0::2], to[0::2])
    r_odd = rel_rows(tg[1::2], to1[1::2]) if K > 1 else np.zeros(1)
    log(f"    even bins max rel {r_even.max():.2e}, odd bins max rel {r_odd.max():.2e}")
    assert r_even.max() <= ROW_TOL and r_odd.max() <= ROW_TOL
    ro = np.sqrt(oracle.tensor_sse(*groupings(M, N, K, ptr, col, bins, val)[0], U, V, tg)
                 / col.size)
    assert abs(rm - ro) <= 1e-5


@pytest.mark.parametrize("D", [1, 7, 16, 20, 33, 64, 100, 128])
def test_time_chain_draw_matches_oracle(D):
    check_chain(300, 200, 30, D, 700 + D, label="small")


@pytest.mark.parametrize("K", [1, 2, 5])
def test_short_chains(K):
    check_chain(120, 90, K, 12, 740 + K, empty_bins=(), empty_last=False, label="short")


@pytest.mark.parametrize("D", [10, 20, 33, 100])
def test_time_chain_with_split_bins_and_batches(D):
    """Few bins with many ratings each: every bin is split into chunks (like the full-size
    bins), and a small workspace forces several batches per parity."""
    if D <= 20:
        ld = 16 if D <= 16 else 20
        slot = 4 * ((ld * (ld + 1) // 2 + ld + 3) // 4 * 4)
    else:
        t = (D + 15) // 16
        slot = 4 * (t * (t + 1) // 2 * 256 + 16 * t)
    tun = dict(hub_threshold=256, chunk=200, workspace_bytes=25 * slot)
    check_chain(400, 300, 8, D, 780 + D, tuning=tun, empty_bins=(2,), deg=(10, 40),
                label="split")


@pytest.mark.parametrize("D", [1, 2, 5, 20, 33, 100, 128])
def test_time_hyper_matches_oracle(D):
    from paper_1108_2580_amd import ALS

    M, N, K = 200, 150, 257
    ptr, col, val, bins, _, _, _ = problem(M, N, K, 2, 800 + D, empty_bins=())
    rng = np.random.default_rng(810 + D)
    T = (np.cumsum(rng.normal(0, 0.05, size=(K, D)), axis=0) + 1.0).astype(np.float32)
    mu0, W0inv = rng.normal(1, 0.1, size=D), spd(rng, D, 0.3)
    beta0, nu0 = 2.0, D + 2.0
    chi2, offd, zmu = bartlett_variates(rng, D, nu0 + K)
    log(f"time hyper D={D}")
    with ALS(M, N, ptr, col, val, D) as als:
        als.set_time_bins(K, bins)
        als.set_nw_prior("time", mu0, beta0, W0inv, nu0)
        mu_g, Lam_g = als.sample_hyper("time", dev(T), dev(chi2, np.float64),
                                       dev(offd, np.float64), dev(zmu, np.float64), check=True)
    mu_g, Lam_g = mu_g.cpu().numpy(), Lam_g.cpu().numpy()
    post = oracle.time_posterior(T, mu0, beta0, W0inv, nu0)
    mu_o, Lam_o = oracle.nw_sample(post[0], post[1], post[2], chi2, offd, zmu)
    eL = np.linalg.norm(Lam_g - Lam_o) / np.linalg.norm(Lam_o)
    em = np.linalg.norm(mu_g - mu_o) / max(np.linalg.norm(mu_o), 1e-30)
    log(f"  rel Lambda {eL:.2e} rel mu {em:.2e}")
    assert eL <= HYPER_TOL and em <= HYPER_TOL


@pytest.mark.parametrize("D", [1, 20, 100])
def test_alpha_matches_oracle(D):
    from paper_1108_2580_amd import ALS

    M, N, K = 300, 200, 30
    ptr, col, val, bins, U, V, T = problem(M, N, K, D, 900 + D)
    by_user, _, _ = groupings(M, N, K, ptr, col, bins, val)
    w0, nu0 = 0.5, 3.0
    chi2 = float(np.random.default_rng(901).chisquare(nu0 + col.size))
    with ALS(M, N, ptr, col, val, D) as als:
        als.set_time_bins(K, bins)
        a_g = als.tensor_sample_alpha(dev(U), dev(V), dev(T), w0, chi2)
    w_s, _ = oracle.alpha_posterior(oracle.tensor_sse(*by_user, U, V, T), col.size, w0, nu0)
    a_o = w_s * chi2
    log(f"alpha D={D}: gpu {a_g:.9e} oracle {a_o:.9e}")
    assert abs(a_g - a_o) <= ALPHA_TOL * a_o


@pytest.mark.parametrize("k,iters", [(1, 2), (2, 1)])
def test_bptf_iterations_teacher_forced(k, iters):
    """BPTF iterations on a config with seeded time bins (alpha, the three hyperparameter
    draws, then items, users and the chain), every step checked against the oracle fed the
    GPU's inputs."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    D = r.D
    K = 50
    bins = workload.time_bins(r.row_ptr, K, workload.time_seed(k), spread=10.0)
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    T0 = np.ones((K, D), dtype=np.float32)
    by_user, by_item, by_bin = groupings(r.M, r.N, K, r.row_ptr, r.col, bins, r.val)
    rng = np.random.default_rng(5150 + k)
    w0, nu_a = 1.0, 2.0
    log(f"bptf iterations {r.name} bins {K}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        als.set_time_bins(K, bins)
        for side in ("users", "items", "time"):
            als.set_nw_prior(side, np.zeros(D) if side != "time" else np.ones(D), 2.0,
                             np.eye(D), D + 1.0)
        U, V, T = dev(U0), dev(V0), dev(T0)
        for it in range(iters):
            Uh, Vh, Th = (x.cpu().numpy() for x in (U, V, T))
            chi2 = float(rng.chisquare(nu_a + r.nnz))
            alpha = als.tensor_sample_alpha(U, V, T, w0, chi2)
            w_s, _ = oracle.alpha_posterior(oracle.tensor_sse(*by_user, Uh, Vh, Th), r.nnz,
                                            w0, nu_a)
            assert abs(alpha - w_s * chi2) <= ALPHA_TOL * alpha
            hyper = {}
            for side, X, n in (("items", V, r.N), ("users", U, r.M), ("time", T, K)):
                Xh = X.cpu().numpy()
                mu0 = np.ones(D) if side == "time" else np.zeros(D)
                chi, offd, zmu = bartlett_variates(rng, D, D + 1.0 + n)
                mu_g, Lam_g = als.sample_hyper(side, X, dev(chi, np.float64),
                                               dev(offd, np.float64), dev(zmu, np.float64),
                                               check=True)
                post = (oracle.time_posterior if side == "time" else oracle.nw_posterior)(
                    Xh, mu0, 2.0, np.eye(D), D + 1.0)
                mu_o, Lam_o = oracle.nw_sample(post[0], post[1], post[2], chi, offd, zmu)
                eL = np.linalg.norm(Lam_g.cpu().numpy() - Lam_o) / np.linalg.norm(Lam_o)
                assert eL <= HYPER_TOL
                hyper[side] = (mu_g, Lam_g)
            for mode, groups, rows in (("items", by_item, r.N), ("users", by_user, r.M),
                                       ("bins", by_bin, K)):
                Uh, Vh, Th = (x.cpu().numpy() for x in (U, V, T))
                mu_g, Lam_g = hyper["time" if mode == "bins" else mode]
                z = rng.standard_normal((rows, D), dtype=np.float32)
                rm = als.tensor_gibbs_half_sweep(mode, U, V, T, alpha, Lam_g, mu_g, dev(z),
                                                 rmse=True)
                p, i1, i2, v = groups
                Lh, mh = Lam_g.cpu().numpy(), mu_g.cpu().numpy()
                if mode == "bins":
                    tg = T.cpu().numpy()
                    to, _ = oracle.time_rows(p, i1, i2, v, Uh, Vh, alpha, Lh, mh, z, 0, Th)
                    te = Th.astype(np.float64).copy()
                    te[0::2] = tg[0::2]
                    to1, _ = oracle.time_rows(p, i1, i2, v, Uh, Vh, alpha, Lh, mh, z, 1, te)
                    rr = np.concatenate([rel_rows(tg[0::2], to[0::2]),
                                         rel_rows(tg[1::2], to1[1::2])])
                else:
                    F1, F2, X = (Vh, Th, Uh) if mode == "users" else (Uh, Th, Vh)
                    xo, fl = oracle.tensor_gibbs_rows(p, i1, i2, v, F1, F2, alpha, Lh, mh, z, X)
                    assert not fl.any()
                    rr = rel_rows((U if mode == "users" else V).cpu().numpy(), xo)
                log(f"  iter {it + 1} {mode}: alpha {alpha:.4f} rows max rel {rr.max():.2e} "
                    f"RMSE {rm:.4f}")
                assert rr.max() <= ROW_TOL


def test_bptf_argument_errors():
    from paper_1108_2580_amd import ALS, ALSError, ALS_ERR_INVALID_ARG

    M, N, K, D = 40, 30, 5, 4
    ptr, col, val, bins, U, V, T = problem(M, N, K, D, 3, empty_bins=())
    Lam, mu = dev(np.eye(D), np.float64), dev(np.zeros(D), np.float64)
    log("bptf argument errors")
    with ALS(M, N, ptr, col, val, D) as als:
        Ud, Vd, Td = dev(U), dev(V), dev(T)
        als.n_bins = K
        with pytest.raises(ALSError) as e:  # no time bins yet
            als.tensor_gibbs_half_sweep("bins", Ud, Vd, Td, 1.0, Lam, mu, dev(np.zeros((K, D))))
        assert e.value.status == ALS_ERR_INVALID_ARG
        als.set_time_bins(K, bins)
        with pytest.raises(ALSError):  # no chain prior
            als.sample_hyper("time", Td, dev(np.ones(D), np.float64),
                             dev(np.zeros(D * (D - 1) // 2), np.float64),
                             dev(np.zeros(D), np.float64))
        with pytest.raises(ALSError):
            als.tensor_gibbs_half_sweep("bins", Ud, Vd, Td, 0.0, Lam, mu, dev(np.zeros((K, D))))
        with pytest.raises(ALSError):
            als.tensor_sample_alpha(Ud, Vd, Td, -1.0, 3.0)
        als.set_weights(np.ones(col.size))
        with pytest.raises(ALSError):
            als.tensor_gibbs_half_sweep("users", Ud, Vd, Td, 1.0, Lam, mu, dev(np.zeros((M, D))))
        als.set_weights(None)
        als.tensor_gibbs_half_sweep("users", Ud, Vd, Td, 1.0, Lam, mu, dev(np.zeros((M, D))))


def sub_chain(p, i1, i2, v, T, k):
    """The bins around bin k (k - 1, k, k + 1 where they exist) with bin k's ratings only,
    and the position of k in it: its conditional is the same as in the whole chain (first
    bin: the mean mu_T; last bin: one neighbour)."""
    K = T.shape[0]
    lo, hi = max(k - 1, 0), min(k + 1, K - 1)
    n = int(p[k + 1] - p[k])
    pos = k - lo
    counts = np.zeros(hi - lo + 1, dtype=np.int64)
    counts[pos] = n
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    sl = slice(p[k], p[k + 1])
    return ptr, i1[sl], i2[sl], v[sl], T[lo:hi + 1], pos


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 4])
def test_full_size_bptf_sampled(k):
    """Full-size workload with 6649 time bins: one draw of each mode from the seeded state
    (the bins even, then odd), checked on sampled users and items (largest, smallest and
    random) and on sampled bins through their neighbourhood sub-chains."""
    from paper_1108_2580_amd import ALS
    from tests.test_gpu_full import sample_rows

    r = workload.make_config(k)
    D = r.D
    K = workload.N_TIME_BINS
    bins = workload.time_bins(r.row_ptr, K, workload.time_seed(3))
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(61 + k)
    T0 = (1.0 + 0.1 * rng.standard_normal((K, D))).astype(np.float32)
    val = r.val.astype(np.float64)
    by_user = (r.row_ptr, r.col, bins, val)
    cp, cu, cv = oracle.transpose(r.row_ptr, r.col, val, r.N)
    _, _, cb = oracle.transpose(r.row_ptr, r.col, bins.astype(np.float64), r.N)
    by_item = (cp, cu, cb.astype(np.int32), cv)
    bp, bu, bv = oracle.transpose(r.row_ptr, bins, val, K)
    _, _, bi = oracle.transpose(r.row_ptr, bins, r.col.astype(np.float64), K)
    by_bin = (bp, bu, bi.astype(np.int32), bv)
    alpha = 1.0 / 900.0
    log(f"full-size bptf {r.name}: {K} bins")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        als.set_time_bins(K, bins)
        for mode, groups, nsamp in (("items", by_item, 256), ("users", by_user, 256)):
            Lam, mu = spd(rng, D, 2.0), rng.normal(0, 0.05, size=D)
            n = r.N if mode == "items" else r.M
            z = rng.standard_normal((n, D), dtype=np.float32)
            U, V, T = dev(U0), dev(V0), dev(T0)
            als.tensor_gibbs_half_sweep(mode, U, V, T, alpha, dev(Lam, np.float64),
                                        dev(mu, np.float64), dev(z))
            assert als.flagged_rows() == 0
            F1, F2, X = (U0, T0, V0) if mode == "items" else (V0, T0, U0)
            xg = (V if mode == "items" else U).cpu().numpy()
            p, i1, i2, v = groups
            rows = sample_rows(p, 9 + k)
            rows = np.unique(np.concatenate([rows[:8], rows[-8:], rows[8:8 + nsamp]]))
            sub_ptr = np.concatenate([[0], np.cumsum(p[rows + 1] - p[rows])]).astype(np.int64)
            take = np.concatenate([np.arange(p[s], p[s + 1]) for s in rows])
            xo, fl = oracle.tensor_gibbs_rows(sub_ptr, i1[take], i2[take], v[take], F1, F2, alpha,
                                              Lam, mu, z[rows], X[rows])
            assert not fl.any()
            rr = rel_rows(xg[rows], xo)
            log(f"  mode={mode}: {rows.size} sampled rows, max rel {rr.max():.2e}")
            assert rr.max() <= ROW_TOL
            assert np.isfinite(xg).all()
        # the chain
        Lam, mu = spd(rng, D, 20.0), 1.0 + rng.normal(0, 0.01, size=D)
        z = rng.standard_normal((K, D), dtype=np.float32)
        U, V, T = dev(U0), dev(V0), dev(T0)
        als.tensor_gibbs_half_sweep("bins", U, V, T, alpha, dev(Lam, np.float64),
                                    dev(mu, np.float64), dev(z))
        assert als.flagged_rows() == 0
        tg = T.cpu().numpy()
    p, i1, i2, v = by_bin
    picks = np.unique(np.concatenate([[0, 1, K - 2, K - 1],
                                      np.random.default_rng(5 + k).choice(K, 40, replace=False)]))
    te = T0.astype(np.float64).copy()
    te[0::2] = tg[0::2]  # the odd bins are drawn given the GPU's even bins
    worst = 0.0
    for b in picks:
        state = T0.astype(np.float64) if b % 2 == 0 else te
        sp, s1, s2, sv, sT, pos = sub_chain(p, i1, i2, v, state, int(b))
        sz = np.zeros((sT.shape[0], D))
        sz[pos] = z[b]
        parity = pos % 2
        to, fl = oracle.time_rows(sp, s1, s2, sv, U0, V0, alpha, Lam, mu, sz, parity, sT)
        assert not fl.any()
        worst = max(worst, float(rel_rows(tg[b:b + 1], to[pos:pos + 1])[0]))
    log(f"  chain: {picks.size} sampled bins, max rel {worst:.2e}")
    assert worst <= ROW_TOL
