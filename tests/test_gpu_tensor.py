"""Tensor ALS over time bins on the GPU (als_set_time_bins, als_tensor_half_sweep,
als_tensor_rmse) against the fp64 oracle.

Bars as for the matrix half-sweep: relative row error <= 1e-4 after one mode update from
identical inputs; rows without ratings and flagged rows untouched; training RMSE within
1e-5 of the oracle's. With all time factors equal to one, a mode update is exactly the
matrix update (f * 1 = f), so the tensor kernels must reproduce the matrix kernels bit
for bit.
"""
import sys

import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROW_TOL = 1e-4
RMSE_TOL = 1e-5


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def rel_rows(x, ref):
    return np.linalg.norm(x - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)


def tensor_problem(M, N, n_bins, D, seed, zero_users=2, deg=(6, 30)):
    rng = np.random.default_rng(seed)
    degs = rng.integers(deg[0], deg[1], size=M)
    degs[rng.choice(M, zero_users, replace=False)] = 0
    ptr, col, val = workload.make_custom(M, N, degs, seed)
    bins = rng.integers(0, n_bins - 1, size=col.size).astype(np.int32)  # bin n_bins-1 empty
    U = rng.normal(0, 0.5, size=(M, D)).astype(np.float32)
    V = rng.normal(0, 0.5, size=(N, D)).astype(np.float32)
    T = rng.normal(1.0, 0.3, size=(n_bins, D)).astype(np.float32)
    return ptr, col, val, bins, U, V, T


def check_modes(M, N, n_bins, ptr, col, val, bins, U, V, T, D, lam, tuning=None, label=""):
    from paper_1108_2580_amd import ALS

    t = oracle.TensorTrajectory(M, N, n_bins, ptr, col, bins, val.astype(np.float64), U, V, T, lam)
    with ALS(M, N, ptr, col, val, D, tuning=tuning) as als:
        als.set_time_bins(n_bins, bins)
        for mode, groups, F1, F2, X in (("users", t.by_user, V, T, U),
                                        ("items", t.by_item, U, T, V),
                                        ("bins", t.by_bin, U, V, T)):
            log(f"  {label} tensor mode={mode} D={D}")
            Ud, Vd, Td = dev(U), dev(V), dev(T)
            rm = als.tensor_half_sweep(mode, Ud, Vd, Td, lam, rmse=True, allow_flagged=True)
            xg = {"users": Ud, "items": Vd, "bins": Td}[mode].cpu().numpy()
            p, i1, i2, v = groups
            xo, fl = oracle.tensor_rows(p, i1, i2, v, F1, F2, lam, X)
            assert als.flagged_rows() == int((fl == 1).sum())
            solved = fl == 0
            r = rel_rows(xg[solved], xo[solved])
            log(f"    rows {solved.sum()} max rel {r.max():.2e}")
            assert r.max() <= ROW_TOL
            assert np.array_equal(xg[~solved], X[~solved])
            # the RMSE of the new state, against the oracle's residual of the GPU's state
            Un, Vn, Tn = (xg if mode == "users" else U, xg if mode == "items" else V,
                          xg if mode == "bins" else T)
            ro = np.sqrt(oracle.tensor_sse(ptr, col, bins, val, Un, Vn, Tn) / col.size)
            assert abs(rm - ro) <= RMSE_TOL


@pytest.mark.parametrize("D", [1, 7, 10, 16, 17, 20, 33, 64, 100, 128])
def test_tensor_modes_match_oracle(D):
    M, N, n_bins = 300, 200, 40
    ptr, col, val, bins, U, V, T = tensor_problem(M, N, n_bins, D, 500 + D)
    check_modes(M, N, n_bins, ptr, col, val, bins, U, V, T, D, 0.065, label="small")


@pytest.mark.parametrize("D", [10, 20, 33, 100])
def test_tensor_split_rows_and_batches(D):
    """Few bins with many ratings each: every time-bin row is split into chunks, and a
    small workspace forces several batches."""
    M, N, n_bins = 400, 300, 6
    ptr, col, val, bins, U, V, T = tensor_problem(M, N, n_bins, D, 800 + D, deg=(10, 40))
    if D <= 20:
        slot = 4 * ((lambda ld: (ld * (ld + 1) // 2 + ld + 3) // 4 * 4)(16 if D <= 16 else 20))
    else:
        t = (D + 15) // 16
        slot = 4 * (t * (t + 1) // 2 * 256 + 16 * t)
    # room for 25 chunk slots: a bin row needs about 10, so the bins take several batches
    tun = dict(hub_threshold=256, chunk=200, workspace_bytes=25 * slot)
    check_modes(M, N, n_bins, ptr, col, val, bins, U, V, T, D, 0.065, tuning=tun, label="split")


def strip_width(D):
    """Widths whose matrix Gram takes the strip form (the last 16-feature tile uses at most
    four features, three or more tiles); the tensor Gram keeps the tile form, so there the
    two sum the last tile column in different orders."""
    T = (D + 15) // 16
    return T >= 3 and D - 16 * (T - 1) <= 4


@pytest.mark.parametrize("D", [20, 64, 100])
def test_unit_time_factors_are_matrix_als(D):
    """Bit for bit where both Grams take the same form; at the strip widths the rows agree
    to fp32 summation-order rounding (relative 1e-5, far inside the 1e-4 bar)."""
    from paper_1108_2580_amd import ALS

    M, N, n_bins = 250, 180, 12
    ptr, col, val, bins, U, V, _ = tensor_problem(M, N, n_bins, D, 900 + D)
    ones = np.ones((n_bins, D), dtype=np.float32)
    exact = not strip_width(D)
    log(f"tensor with unit time factors D={D} exact={exact}")
    with ALS(M, N, ptr, col, val, D) as als:
        als.set_time_bins(n_bins, bins)
        for mode, side, fixed, X in (("users", "users", V, U), ("items", "items", U, V)):
            Ud, Vd, Td = dev(U), dev(V), dev(ones)
            als.tensor_half_sweep(mode, Ud, Vd, Td, 0.065)
            xt = (Ud if mode == "users" else Vd).cpu().numpy()
            out = dev(X)
            als.half_sweep(side, dev(fixed), 0.065, out)
            xm = out.cpu().numpy()
            if exact:
                assert np.array_equal(xt, xm)
            else:
                assert rel_rows(xt, xm).max() <= 1e-5
        r_t = als.tensor_rmse(dev(U), dev(V), dev(ones))
        r_m = als.rmse(dev(U), dev(V))
        assert r_t == r_m


def test_tensor_free_running_config1():
    """Three sweeps (items, users, bins) of config 1 with seeded time bins; the training
    RMSE after every mode update within 1e-5 of the free-running fp64 oracle."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(1)
    n_bins = 50
    bins = workload.time_bins(r.row_ptr, n_bins, workload.time_seed(1), spread=10.0)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    T0 = np.ones((n_bins, r.D), dtype=np.float32)
    t = oracle.TensorTrajectory(r.M, r.N, n_bins, r.row_ptr, r.col, bins,
                                r.val.astype(np.float64), U0, V0, T0, r.lam)
    log(f"tensor free running {r.name} bins {n_bins}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        als.set_time_bins(n_bins, bins)
        U, V, T = dev(U0), dev(V0), dev(T0)
        for s in range(3):
            for mode in ("items", "users", "bins"):
                g = als.tensor_half_sweep(mode, U, V, T, r.lam, rmse=True)
                t.step(mode)
                o = t.rmse()
                log(f"  sweep {s + 1} {mode}: RMSE gpu {g:.7f} oracle {o:.7f} diff {g - o:.2e}")
                assert abs(g - o) <= RMSE_TOL


def test_tensor_argument_errors():
    from paper_1108_2580_amd import ALS, ALSError, ALS_ERR_INVALID_ARG

    M, N, n_bins, D = 40, 30, 5, 4
    ptr, col, val, bins, U, V, T = tensor_problem(M, N, n_bins, D, 3)
    log("tensor argument errors")
    with ALS(M, N, ptr, col, val, D) as als:
        Ud, Vd = dev(U), dev(V)
        als.n_bins = n_bins
        with pytest.raises(ALSError) as e:
            als.tensor_half_sweep("users", Ud, Vd, dev(T), 0.1)
        assert e.value.status == ALS_ERR_INVALID_ARG
        bad = bins.copy()
        bad[3] = n_bins
        with pytest.raises(ALSError):
            als.set_time_bins(n_bins, bad)
        bad[3] = -1
        with pytest.raises(ALSError):
            als.set_time_bins(n_bins, bad)
        # the staged time-bin table, (n_bins + 1) rows of 16 * ceil(D / 16) floats, must stay
        # below 4 GiB; at n_bins = 2^31 - 1 the row count is formed in 64 bits, and the call
        # is refused before it reads a bin
        for nb in (2**31 - 1, 2**26 - 1):
            with pytest.raises(ALSError) as e:
                als.set_time_bins(nb, bins)
            assert e.value.status == ALS_ERR_INVALID_ARG and "limit" in str(e.value)
        als.set_time_bins(n_bins, bins)
        Td = dev(T)
        with pytest.raises(ALSError):  # U and V the same buffer
            als.tensor_half_sweep("users", Ud, Ud[: N], Td, 0.1)
        als.set_weights(np.ones(col.size))
        with pytest.raises(ALSError):
            als.tensor_half_sweep("users", Ud, Vd, Td, 0.1)
        als.set_weights(None)
        als.tensor_half_sweep("users", Ud, Vd, Td, 0.1)


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 4])
def test_full_size_tensor_sampled_rows(k):
    """Full-size workload with the paper's 6649 time bins: one update of each mode from the
    seeded factors (T = 1 + noise), checked on sampled rows of the mode. Every mode starts
    from the seeded state, as the per-row bar is stated for the first update; after an
    update the other modes' systems can be far worse conditioned."""
    from paper_1108_2580_amd import ALS
    from tests.test_gpu_full import sample_rows

    r = workload.make_config(k)
    D = r.D
    nb = workload.N_TIME_BINS
    bins = workload.time_bins(r.row_ptr, nb, workload.time_seed(3))
    U0, V0 = workload.init_factors(r.M, r.N, D, r.init_seed)
    rng = np.random.default_rng(31 + k)
    T0 = (1.0 + 0.1 * rng.standard_normal((nb, D))).astype(np.float32)
    val = r.val.astype(np.float64)
    # the three groupings through the oracle's own transpose (payloads carried along)
    by_user = (r.row_ptr, r.col, bins, val)
    cp, cu, cv = oracle.transpose(r.row_ptr, r.col, val, r.N)
    _, _, cb = oracle.transpose(r.row_ptr, r.col, bins.astype(np.float64), r.N)
    by_item = (cp, cu, cb.astype(np.int32), cv)
    bp, bu, bv = oracle.transpose(r.row_ptr, bins, val, nb)
    _, _, bi = oracle.transpose(r.row_ptr, bins, r.col.astype(np.float64), nb)
    by_bin = (bp, bu, bi.astype(np.int32), bv)
    log(f"full-size tensor {r.name}: {nb} bins")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, D) as als:
        als.set_time_bins(nb, bins)
        for mode, groups, nsamp in (("items", by_item, 256), ("users", by_user, 256),
                                    ("bins", by_bin, 24)):
            U, V, T = dev(U0), dev(V0), dev(T0)
            F = {"users": (V, T, U), "items": (U, T, V), "bins": (U, V, T)}[mode]
            F1, F2, X = (a.cpu().numpy() for a in F)
            als.tensor_half_sweep(mode, U, V, T, r.lam)
            assert als.flagged_rows() == 0
            xg = F[2].cpu().numpy()
            p, i1, i2, v = groups
            rows = sample_rows(p, 7 + k)
            rows = np.unique(np.concatenate([rows[:8], rows[-8:], rows[8:8 + nsamp]]))
            sub_ptr = np.concatenate([[0], np.cumsum(p[rows + 1] - p[rows])]).astype(np.int64)
            take = np.concatenate([np.arange(p[s], p[s + 1]) for s in rows])
            xo, fl = oracle.tensor_rows(sub_ptr, i1[take], i2[take], v[take], F1, F2, r.lam,
                                        X[rows])
            assert not fl.any()
            rr = rel_rows(xg[rows], xo)
            log(f"  mode={mode}: {rows.size} sampled rows, max rel {rr.max():.2e}")
            assert rr.max() <= ROW_TOL
            assert np.isfinite(xg).all()
