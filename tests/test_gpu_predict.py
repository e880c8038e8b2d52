"""Held-out predictions and validation RMSE on the GPU (als_predict, als_set_holdout,
als_holdout_rmse) against the fp64 oracle, element by element.

Tolerance, derived from the arithmetic: the kernel forms u . v as a chain of D fused
multiply-adds in fp32 (one rounding each), so |r_hat_gpu - u . v| <= gamma_D * S with
gamma_D = D u / (1 - D u), u = 2^-24 and S = sum_k |u_k v_k|; the fp64 oracle is within
D 2^-53 S of the exact value. Every prediction is checked against the sum of the two
bounds. The validation RMSE differs from the oracle's by at most the root mean square
of the per-pair bounds (triangle inequality in the 2-norm), and by at most 1e-5.
"""
import sys

import numpy as np
import pytest

import oracle
import workload

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

RMSE_TOL = 1e-5


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_f(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


def dev_i(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda:0")


def pred_bound(U, V, users, items):
    """Per-pair bound on |r_hat_gpu - r_hat_oracle|."""
    D = U.shape[1]
    S = np.empty(len(users))
    for a in range(0, len(users), 1 << 20):
        b = a + (1 << 20)
        S[a:b] = np.abs(U[users[a:b]].astype(np.float64) * V[items[a:b]]).sum(axis=1)
    u = 2.0 ** -24
    return (D * u / (1 - D * u) + D * 2.0 ** -53) * S * 1.0001 + 1e-45


def small_ctx(M, N, D, seed=0):
    from paper_1108_2580_amd import ALS

    ptr, col, val = workload.make_custom(M, N, np.full(M, 3), seed)
    return ALS(M, N, ptr, col, val, D)


@pytest.mark.parametrize("D", [1, 2, 3, 4, 7, 8, 10, 16, 20, 33, 64, 100, 127, 128])
def test_predict_matches_oracle(D):
    M, N, n = 300, 200, 10_007
    rng = np.random.default_rng(100 + D)
    U = rng.standard_normal((M, D), dtype=np.float32)
    V = rng.standard_normal((N, D), dtype=np.float32)
    users = rng.integers(0, M, n).astype(np.int32)
    items = rng.integers(0, N, n).astype(np.int32)
    log(f"predict D={D} n={n}")
    with small_ctx(M, N, D) as als:
        got = als.predict(dev_f(U), dev_f(V), dev_i(users), dev_i(items)).cpu().numpy()
    want = oracle.predict(users, items, U, V)
    err = np.abs(got.astype(np.float64) - want)
    bound = pred_bound(U, V, users, items)
    log(f"  max err/bound {np.max(err / bound):.3f}")
    assert np.all(err <= bound)


@pytest.mark.parametrize("n", [0, 1, 63, 255, 256, 257, 4099])
def test_predict_sizes(n):
    M, N, D = 50, 40, 20
    rng = np.random.default_rng(n)
    U = rng.standard_normal((M, D), dtype=np.float32)
    V = rng.standard_normal((N, D), dtype=np.float32)
    users = rng.integers(0, M, n).astype(np.int32)
    items = rng.integers(0, N, n).astype(np.int32)
    log(f"predict sizes n={n}")
    with small_ctx(M, N, D) as als:
        out = torch.full((n + 64,), 7.0, device="cuda:0")
        als.predict(dev_f(U), dev_f(V), dev_i(users), dev_i(items), out=out[:n])
        o = out.cpu().numpy()
    assert np.all(o[n:] == 7.0), "wrote past the end of pred"
    want = oracle.predict(users, items, U, V)
    assert np.all(np.abs(o[:n] - want) <= pred_bound(U, V, users, items))


def test_predict_out_of_range_pairs_give_nan():
    M, N, D = 30, 20, 12
    rng = np.random.default_rng(5)
    U = rng.standard_normal((M, D), dtype=np.float32)
    V = rng.standard_normal((N, D), dtype=np.float32)
    users = rng.integers(0, M, 600).astype(np.int32)
    items = rng.integers(0, N, 600).astype(np.int32)
    bad = np.zeros(600, dtype=bool)
    for k, (uu, ii) in enumerate([(-1, 0), (M, 0), (0, N), (0, -5), (2**31 - 1, 3),
                                  (-2**31, -2**31)]):
        users[50 * k + 7], items[50 * k + 7] = uu, ii
        bad[50 * k + 7] = True
    log("predict out-of-range pairs")
    with small_ctx(M, N, D) as als:
        got = als.predict(dev_f(U), dev_f(V), dev_i(users), dev_i(items)).cpu().numpy()
    assert np.all(np.isnan(got[bad]))
    ok = ~bad
    want = oracle.predict(users[ok], items[ok], U, V)
    assert np.all(np.abs(got[ok] - want) <= pred_bound(U, V, users[ok], items[ok]))


def test_predict_argument_errors():
    from paper_1108_2580_amd import ALSError, ALS_ERR_INVALID_ARG, lib
    import ctypes

    M, N, D = 10, 8, 4
    U = dev_f(np.ones((M, D)))
    V = dev_f(np.ones((N, D)))
    ix = dev_i(np.zeros(4))
    log("predict argument errors")
    with small_ctx(M, N, D) as als:
        with pytest.raises(ALSError) as e:
            als.predict(U, V, ix, ix, out=U.view(-1)[:4])
        assert e.value.status == ALS_ERR_INVALID_ARG
        st = lib.als_predict(als._h, ctypes.c_void_p(U.data_ptr() + 4), ctypes.c_void_p(V.data_ptr()),
                             4, ctypes.c_void_p(ix.data_ptr()), ctypes.c_void_p(ix.data_ptr()),
                             ctypes.c_void_p(torch.empty(4, device="cuda:0").data_ptr()))
        assert st == ALS_ERR_INVALID_ARG
        assert lib.als_predict(als._h, None, None, -1, None, None, None) == ALS_ERR_INVALID_ARG
        assert lib.als_predict(als._h, None, None, 0, None, None, None) == 0


@pytest.mark.parametrize("D", [10, 20, 33, 100])
def test_holdout_rmse_matches_oracle(D):
    M, N, n = 500, 300, 20_011
    rng = np.random.default_rng(200 + D)
    U = (rng.standard_normal((M, D)) * (7.0 / np.sqrt(D))).astype(np.float32)
    V = (rng.standard_normal((N, D)) * (7.0 / np.sqrt(D)) + 0.5).astype(np.float32)
    users = rng.integers(0, M, n).astype(np.int32)
    items = rng.integers(0, N, n).astype(np.int32)
    r = rng.integers(0, 101, n).astype(np.uint8)
    log(f"holdout rmse D={D}")
    with small_ctx(M, N, D) as als:
        als.set_holdout(users, items, r)
        Ud, Vd = dev_f(U), dev_f(V)
        got = als.holdout_rmse(Ud, Vd)
        again = als.holdout_rmse(Ud, Vd)
    want = oracle.pair_rmse(users, items, r.astype(np.float64), U, V)
    bound = np.sqrt(np.mean(pred_bound(U, V, users, items) ** 2)) + 1e-12 * want
    log(f"  gpu {got!r} oracle {want!r} diff {got - want:.3e} bound {bound:.3e}")
    assert got == again, "not reproducible"
    assert abs(got - want) <= min(bound, RMSE_TOL)


def test_holdout_registration():
    from paper_1108_2580_amd import ALSError, ALS_ERR_INVALID_ARG

    M, N, D = 40, 30, 8
    rng = np.random.default_rng(9)
    U = rng.standard_normal((M, D), dtype=np.float32)
    V = rng.standard_normal((N, D), dtype=np.float32)
    log("holdout registration")
    with small_ctx(M, N, D) as als:
        Ud, Vd = dev_f(U), dev_f(V)
        with pytest.raises(ALSError) as e:
            als.holdout_rmse(Ud, Vd)
        assert e.value.status == ALS_ERR_INVALID_ARG
        for uu, ii in ((M, 0), (-1, 0), (0, N), (0, -1)):
            with pytest.raises(ALSError) as e:
                als.set_holdout([0, uu], [1, ii], [3, 4])
            assert e.value.status == ALS_ERR_INVALID_ARG
        als.set_holdout([], [], [])
        assert als.holdout_rmse(Ud, Vd) == 0.0
        # a replacement set, given out of user order, with a duplicate pair
        users = np.array([5, 2, 5, 39, 0, 2], dtype=np.int32)
        items = np.array([1, 29, 1, 0, 7, 3], dtype=np.int32)
        r = np.array([10, 0, 30, 100, 55, 1], dtype=np.uint8)
        als.set_holdout(users, items, r)
        got = als.holdout_rmse(Ud, Vd)
    want = oracle.pair_rmse(users, items, r.astype(np.float64), U, V)
    assert abs(got - want) <= min(np.sqrt(np.mean(pred_bound(U, V, users, items) ** 2)), RMSE_TOL)


@pytest.mark.parametrize("k,frac,sweeps", [(1, 0.1, 5), (2, 0.02, 3)])
def test_validation_rmse_free_running(k, frac, sweeps):
    """The validation protocol of Sec. 4.1 on a seeded split: train on the rest, report the
    held-out RMSE after every sweep. Two checks per sweep:
    - the GPU's validation RMSE of its own state against the oracle's evaluation of that
      same state, within the arithmetic bound of the module docstring (and 1e-5);
    - the free-running GPU trajectory against the free-running fp64 oracle trajectory,
      within 1e-5 relative: a held-out prediction extrapolates from the two factor rows,
      so it carries their relative error (fp32 factors, per-row bar 1e-4) rather than an
      absolute one, and the held-out RMSE of an overfitting model can be several times
      the training RMSE."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    tp, tc, tv, hu, hi, hr = workload.holdout_split(r.row_ptr, r.col, r.val, frac,
                                                    workload.holdout_seed(k), min_keep=2)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    log(f"validation protocol {r.name}: train {tp[-1]} held out {hu.size} sweeps {sweeps}")
    t = oracle.Trajectory(r.M, r.N, tp, tc, tv.astype(np.float64), U0, V0, r.lam)
    hrf = hr.astype(np.float64)
    with ALS(r.M, r.N, tp, tc, tv, r.D) as als:
        als.set_holdout(hu, hi, hr)
        U, V = dev_f(U0), dev_f(V0)
        g0 = als.holdout_rmse(U, V)
        assert abs(g0 - oracle.pair_rmse(hu, hi, hrf, U0, V0)) <= RMSE_TOL
        for s in range(sweeps):
            als.half_sweep("items", U, r.lam, V)
            als.half_sweep("users", V, r.lam, U)
            t.sweep()
            g = als.holdout_rmse(U, V)
            Ug, Vg = U.cpu().numpy(), V.cpu().numpy()
            same = oracle.pair_rmse(hu, hi, hrf, Ug, Vg)
            o = oracle.pair_rmse(hu, hi, hrf, t.U, t.V)
            bound = np.sqrt(np.mean(pred_bound(Ug, Vg, hu, hi) ** 2)) + 1e-12 * same
            log(f"  sweep {s + 1}: validation RMSE gpu {g:.7f}, oracle on the GPU state "
                f"{same:.7f} (diff {g - same:.2e}, bound {bound:.2e}), oracle trajectory "
                f"{o:.7f} (rel diff {(g - o) / o:.2e}); training RMSE {t.rmse():.4f}")
            assert abs(g - same) <= min(bound, RMSE_TOL)
            assert abs(g - o) <= 1e-5 * o


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 4])
def test_full_size_heldout_pairs(k):
    """Full-size workload: every prediction of 1/64 of the stored positions against the
    oracle, and the validation RMSE of the same pairs."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    users, items, rat = workload.stored_pairs(r.row_ptr, r.col, r.val, r.nnz // 64,
                                              workload.holdout_seed(k))
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    # factors of realistic magnitude: one half-sweep each way from the seeded init
    log(f"full-size held-out pairs {r.name}: {users.size} pairs")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        U, V = dev_f(U0), dev_f(V0)
        als.half_sweep("items", U, r.lam, V)
        als.half_sweep("users", V, r.lam, U)
        got = als.predict(U, V, dev_i(users), dev_i(items)).cpu().numpy()
        als.set_holdout(users, items, rat)
        rm = als.holdout_rmse(U, V)
        Uh, Vh = U.cpu().numpy(), V.cpu().numpy()
    want = oracle.predict(users, items, Uh, Vh)
    bound = pred_bound(Uh, Vh, users, items)
    err = np.abs(got.astype(np.float64) - want)
    log(f"  max err/bound {np.max(err / bound):.3f}; max |pred| {np.abs(want).max():.3f}")
    assert np.all(err <= bound)
    ro = oracle.pair_rmse(users, items, rat.astype(np.float64), Uh, Vh)
    log(f"  validation RMSE gpu {rm!r} oracle {ro!r}")
    assert abs(rm - ro) <= min(np.sqrt(np.mean(bound ** 2)) + 1e-12 * ro, RMSE_TOL)
