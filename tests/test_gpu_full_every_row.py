"""Every row at full size, D = 20, for the methods beside plain ALS: weighted ALS, the BPMF
Gibbs draws, tensor ALS and BPTF. One update of each side or mode from the seeded state,
with the same variates on both sides, every row against the fp64 oracle at the
half-sweep's bar (relative row error 1e-4). The wider widths are covered on sampled rows
in the per-method modules."""
import sys

import numpy as np
import pytest

import oracle
import workload

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
torch = pytest.importorskip("torch")

ROW_TOL = 1e-4


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a, dtype=np.float32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).to("cuda:0")


def check(label, xg, xo, prev, has):
    rel = (np.linalg.norm(xg[has] - xo[has], axis=1)
           / np.maximum(np.linalg.norm(xo[has], axis=1), 1e-30))
    log(f"  {label}: {has.sum()} rows, rel p50={np.median(rel):.2e} "
        f"p99={np.percentile(rel, 99):.2e} max={rel.max():.2e}")
    assert rel.max() <= ROW_TOL
    assert np.isfinite(xg).all()


def spd(rng, D, scale):
    A = rng.normal(size=(D, D))
    return scale * (A @ A.T / D + np.eye(D))


def test_weighted_every_row():
    from paper_1108_2580_amd import ALS

    r = workload.make_config(3)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    w = workload.rating_weights(r.nnz, workload.weight_seed(3)).astype(np.float64)
    val = r.val.astype(np.float64)
    cp, ci, cv = oracle.transpose(r.row_ptr, r.col, val, r.N)
    _, _, cw = oracle.transpose(r.row_ptr, r.col, w, r.N)
    log(f"weighted ALS, every row of {r.name}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        als.set_weights(w.astype(np.float32))
        for side, fixed, prev, (p, i, v, ww) in (("items", U0, V0, (cp, ci, cv, cw)),
                                                 ("users", V0, U0, (r.row_ptr, r.col, val, w))):
            out = dev(prev)
            als.half_sweep(side, dev(fixed), r.lam, out)
            assert als.flagged_rows() == 0
            xo, fl = oracle.half_sweep(p, i, v, fixed, r.lam, prev, w=ww)
            assert not (fl == 1).any()
            check(side, out.cpu().numpy(), xo, prev, np.diff(p) > 0)


def test_gibbs_every_row():
    from paper_1108_2580_amd import ALS

    r = workload.make_config(3)
    D = r.D
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(303)
    alpha = 1.0 / 25.0
    val = r.val.astype(np.float64)
    csc = oracle.transpose(r.row_ptr, r.col, val, r.N)
    log(f"BPMF Gibbs draws, every row of {r.name}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        for side, fixed, prev, (p, i, v), n in (("items", U0, V0, csc, r.N),
                                                ("users", V0, U0, (r.row_ptr, r.col, val), r.M)):
            Lam, mu = spd(rng, D, 2.0), rng.normal(0, 0.05, size=D)
            z = rng.standard_normal((n, D), dtype=np.float32)
            out = dev(prev)
            als.gibbs_half_sweep(side, dev(fixed), alpha, dev(Lam, np.float64),
                                 dev(mu, np.float64), dev(z), out)
            assert als.flagged_rows() == 0
            xo, fl = oracle.gibbs_rows(p, i, v, fixed, alpha, Lam, mu, z, prev)
            assert not fl.any()
            check(side, out.cpu().numpy(), xo, prev, np.ones(n, dtype=bool))


def tensor_groupings(r, bins, K):
    val = r.val.astype(np.float64)
    by_user = (r.row_ptr, r.col, bins, val)
    cp, cu, cv = oracle.transpose(r.row_ptr, r.col, val, r.N)
    _, _, cb = oracle.transpose(r.row_ptr, r.col, bins.astype(np.float64), r.N)
    by_item = (cp, cu, cb.astype(np.int32), cv)
    bp, bu, bv = oracle.transpose(r.row_ptr, bins, val, K)
    _, _, bi = oracle.transpose(r.row_ptr, bins, r.col.astype(np.float64), K)
    by_bin = (bp, bu, bi.astype(np.int32), bv)
    return by_user, by_item, by_bin


def test_tensor_every_row():
    from paper_1108_2580_amd import ALS

    r = workload.make_config(3)
    D, K = r.D, workload.N_TIME_BINS
    bins = workload.time_bins(r.row_ptr, K, workload.time_seed(3))
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    T0 = (1.0 + 0.1 * np.random.default_rng(305).standard_normal((K, D))).astype(np.float32)
    by_user, by_item, by_bin = tensor_groupings(r, bins, K)
    log(f"tensor ALS, every row of {r.name} and every one of {K} bins")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        als.set_time_bins(K, bins)
        for mode, groups in (("items", by_item), ("users", by_user), ("bins", by_bin)):
            U, V, T = dev(U0), dev(V0), dev(T0)
            F1, F2, X = {"users": (V0, T0, U0), "items": (U0, T0, V0),
                         "bins": (U0, V0, T0)}[mode]
            als.tensor_half_sweep(mode, U, V, T, r.lam)
            assert als.flagged_rows() == 0
            xg = {"users": U, "items": V, "bins": T}[mode].cpu().numpy()
            p, i1, i2, v = groups
            xo, fl = oracle.tensor_rows(p, i1, i2, v, F1, F2, r.lam, X)
            assert not (fl == 1).any()
            check(mode, xg, xo, X, np.diff(p) > 0)


def test_bptf_every_row():
    from paper_1108_2580_amd import ALS

    r = workload.make_config(3)
    D, K = r.D, workload.N_TIME_BINS
    bins = workload.time_bins(r.row_ptr, K, workload.time_seed(3))
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(307)
    T0 = (1.0 + 0.1 * rng.standard_normal((K, D))).astype(np.float32)
    by_user, by_item, by_bin = tensor_groupings(r, bins, K)
    alpha = 1.0 / 900.0
    log(f"BPTF draws, every row of {r.name} and every one of {K} bins")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        als.set_time_bins(K, bins)
        for mode, groups, n in (("items", by_item, r.N), ("users", by_user, r.M)):
            Lam, mu = spd(rng, D, 2.0), rng.normal(0, 0.05, size=D)
            z = rng.standard_normal((n, D), dtype=np.float32)
            U, V, T = dev(U0), dev(V0), dev(T0)
            als.tensor_gibbs_half_sweep(mode, U, V, T, alpha, dev(Lam, np.float64),
                                        dev(mu, np.float64), dev(z))
            assert als.flagged_rows() == 0
            F1, F2, X = (U0, T0, V0) if mode == "items" else (V0, T0, U0)
            xg = (V if mode == "items" else U).cpu().numpy()
            p, i1, i2, v = groups
            xo, fl = oracle.tensor_gibbs_rows(p, i1, i2, v, F1, F2, alpha, Lam, mu, z, X)
            assert not fl.any()
            check(mode, xg, xo, X, np.ones(n, dtype=bool))
        # the chain: even bins from the seeded state, odd bins given the GPU's even bins
        Lam, mu = spd(rng, D, 20.0), 1.0 + rng.normal(0, 0.01, size=D)
        z = rng.standard_normal((K, D), dtype=np.float32)
        U, V, T = dev(U0), dev(V0), dev(T0)
        als.tensor_gibbs_half_sweep("bins", U, V, T, alpha, dev(Lam, np.float64),
                                    dev(mu, np.float64), dev(z))
        assert als.flagged_rows() == 0
        tg = T.cpu().numpy()
    p, i1, i2, v = by_bin
    to, fl0 = oracle.time_rows(p, i1, i2, v, U0, V0, alpha, Lam, mu, z, 0, T0)
    te = T0.astype(np.float64).copy()
    te[0::2] = tg[0::2]
    to1, fl1 = oracle.time_rows(p, i1, i2, v, U0, V0, alpha, Lam, mu, z, 1, te)
    assert not fl0.any() and not fl1.any()
    xo = to.copy()
    xo[1::2] = to1[1::2]
    check("bins", tg, xo, T0, np.ones(K, dtype=bool))
