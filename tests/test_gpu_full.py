"""Full-size workloads (the half-sweep at the shapes bench.py times), checked against the
fp64 oracle on sampled rows (the oracle solves them one by one) and on properties that
hold at any size.

Sampled rows per side: the 16 largest (split rows included), the 16 smallest and 224
seeded random rows. Bars as in the small tests: relative row error <= 1e-4 after one
half-sweep from the seeded initial factors; the RMSE returned with the half-sweep equals
the fp64 residual of the GPU state within 1e-5; no row flagged; every factor finite.
"""
import hashlib
import json
import os
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


def sample_rows(ptr, seed):
    deg = np.diff(ptr)
    rows = np.flatnonzero(deg > 0)
    order = rows[np.argsort(-deg[rows], kind="stable")]
    rng = np.random.default_rng(seed)
    pick = np.concatenate([order[:16], order[-16:], rng.choice(rows, 224, replace=False)])
    return np.unique(pick)


@pytest.mark.parametrize("k", [3, 4, 5])
def test_full_first_half_sweep_sampled(k):
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    log(f"{r.name}: nnz={r.nnz} D={r.D}")
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    val = r.val.astype(np.float64)
    csc = oracle.transpose(r.row_ptr, r.col, val, r.N)
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        log(f"  plans users {als.plan_stats('users')} items {als.plan_stats('items')}")
        for side, fixed, prev, (p, i, v) in (("items", U0, V0, csc),
                                             ("users", V0, U0, (r.row_ptr, r.col, val))):
            out = dev(prev)
            rm = als.half_sweep(side, dev(fixed), r.lam, out, rmse=True)
            assert als.flagged_rows() == 0
            xg = out.cpu().numpy()
            assert np.isfinite(xg).all()
            rows = sample_rows(p, seed=k)
            xo, fl = oracle.solve_rows(rows, p, i, v, fixed, r.lam)
            assert (fl == 0).all()
            rel = np.linalg.norm(xg[rows] - xo, axis=1) / np.linalg.norm(xo, axis=1)
            log(f"  {side}: {rows.size} sampled rows (max degree {np.diff(p)[rows].max()}), "
                f"rel p50={np.median(rel):.2e} max={rel.max():.2e}")
            assert rel.max() <= ROW_TOL
            if side == "items":
                ro = oracle.rmse(r.row_ptr, r.col, val, U0, xg)
            else:
                ro = oracle.rmse(r.row_ptr, r.col, val, xg, V0)
            log(f"  {side}: rmse gpu {rm:.9f} oracle on the GPU state {ro:.9f}")
            assert abs(rm - ro) <= RMSE_TOL


def every_row_check(k):
    """One half-sweep per side from the seeded factors at full size, every row against the
    oracle's solve of the same row (p50, p99 and max of the relative row error)."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    val = r.val.astype(np.float64)
    csc = oracle.transpose(r.row_ptr, r.col, val, r.N)
    log(f"every row of {r.name}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        for side, fixed, prev, (p, i, v) in (("items", U0, V0, csc),
                                             ("users", V0, U0, (r.row_ptr, r.col, val))):
            out = dev(prev)
            als.half_sweep(side, dev(fixed), r.lam, out)
            assert als.flagged_rows() == 0
            xg = out.cpu().numpy()
            log(f"  {side}: oracle half-sweep of {p.size - 1} rows ...")
            xo, fl = oracle.half_sweep(p, i, v, fixed, r.lam, prev)
            assert not (fl == 1).any()
            has = np.diff(p) > 0
            rel = (np.linalg.norm(xg[has] - xo[has], axis=1)
                   / np.maximum(np.linalg.norm(xo[has], axis=1), 1e-30))
            log(f"  {side}: {has.sum()} rows, rel p50={np.median(rel):.2e} "
                f"p99={np.percentile(rel, 99):.2e} max={rel.max():.2e}")
            assert rel.max() <= ROW_TOL
            assert np.array_equal(xg[~has], prev[~has])


@pytest.mark.slow
def test_full_d20_every_row():
    every_row_check(3)


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_full_d100_every_row():
    every_row_check(4)


@pytest.mark.slow
@pytest.mark.timeout(1500)
def test_full_d20_free_running_rmse():
    """Five free-running sweeps at full size, D = 20: GPU fp32 vs oracle fp64 trajectory."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(3)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    t = oracle.Trajectory(r.M, r.N, r.row_ptr, r.col, r.val, U0, V0, r.lam)
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        U, V = dev(U0), dev(V0)
        for sweep in range(1, r.sweeps + 1):
            als.half_sweep("items", U, r.lam, V)
            rm = als.half_sweep("users", V, r.lam, U, rmse=True)
            t.sweep()
            ro = t.rmse()
            log(f"  sweep {sweep}: gpu {rm:.9f} oracle {ro:.9f} diff {rm - ro:.2e}")
        assert abs(rm - ro) <= RMSE_TOL


def stored_trajectory(k):
    """The oracle's trajectory of workload k, written by tests/golden/make_wide_trajectories.py
    (oracle and workload only), with the SHA-256 of the inputs it was computed from."""
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                           "wide_trajectories.json")) as f:
        return json.load(f)[str(k)]


@pytest.mark.slow
@pytest.mark.timeout(600)
@pytest.mark.parametrize("k", [4, 5])
def test_full_wide_free_running_rmse(k):
    """Three free-running sweeps at full size, D = 100 and D = 128 (the hub workload): the
    GPU fp32 trajectory against the fp64 oracle's, the training RMSE after every half-sweep
    within 1e-5 (paper Sec. 2.2 for the alternation, Sec. 4.1 for the RMSE). The oracle's
    trajectory is stored with the digests of its inputs; the test first checks that the
    generator still produces exactly those bytes."""
    from paper_1108_2580_amd import ALS

    want = stored_trajectory(k)
    r = workload.make_config(k)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    for name, a in (("row_ptr", r.row_ptr), ("col", r.col), ("val", r.val), ("U0", U0),
                    ("V0", V0)):
        got = hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
        assert got == want["sha256"][name], f"{name} differs from the stored trajectory's input"
    assert (r.D, r.lam, r.sweeps) == (want["D"], want["lambda"], want["sweeps"])
    log(f"wide free running {r.name}, {r.sweeps} sweeps, against the stored oracle trajectory")
    worst = 0.0
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        U, V = dev(U0), dev(V0)
        for sweep in range(r.sweeps):
            for side, fixed, out in (("items", U, V), ("users", V, U)):
                rm = als.half_sweep(side, fixed, r.lam, out, rmse=True)
                assert als.flagged_rows() == 0
                ro = want[f"rmse_after_{side}"][sweep]
                log(f"  sweep {sweep + 1} {side}: gpu {rm:.9f} oracle {ro:.9f} diff {rm - ro:.2e}")
                worst = max(worst, abs(rm - ro))
    log(f"  worst |diff| {worst:.2e}")
    assert worst <= RMSE_TOL


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 5])
def test_full_csc_bit_exact(k):
    """The device CSC at full size (262.8M ratings; the hub workload with 101 columns of
    500,000 ratings) equals the oracle's counting transpose element by element: both
    directions of the alternation (paper Sec. 2.2) read the same ratings."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    log(f"full-size csc {r.name}")
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        got_ptr, got_idx, got_val = als.csc()
    want_ptr, want_idx, want_val = oracle.transpose(r.row_ptr, r.col, r.val.astype(np.float64),
                                                    r.N)
    assert np.array_equal(got_ptr, want_ptr)
    assert np.array_equal(got_idx, want_idx)
    assert np.array_equal(got_val, want_val.astype(np.uint8))
    assert np.array_equal(got_val.astype(np.float64), want_val)
    log(f"  {r.nnz} entries equal; largest column {np.diff(got_ptr).max()}")


@pytest.mark.parametrize("k", [3, 4])
def test_full_weighted_first_half_sweep_sampled(k):
    """Weighted ALS at full size: seeded per-rating weights (log-uniform on [0.25, 4)), one
    half-sweep per side from the seeded factors, sampled rows against the oracle's weighted
    solve (the weights travel to the item side with the oracle's own transpose)."""
    from paper_1108_2580_amd import ALS

    r = workload.make_config(k)
    w = workload.rating_weights(r.nnz, workload.weight_seed(k))
    log(f"{r.name} weighted: nnz={r.nnz} D={r.D}")
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    val = r.val.astype(np.float64)
    w64 = w.astype(np.float64)
    csc = oracle.transpose(r.row_ptr, r.col, val, r.N)
    w_t = oracle.transpose(r.row_ptr, r.col, w64, r.N)[2]
    with ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
        als.set_weights(w)
        for side, fixed, prev, (p, i, v), ww in (("items", U0, V0, csc, w_t),
                                                 ("users", V0, U0, (r.row_ptr, r.col, val), w64)):
            out = dev(prev)
            als.half_sweep(side, dev(fixed), r.lam, out)
            assert als.flagged_rows() == 0
            xg = out.cpu().numpy()
            assert np.isfinite(xg).all()
            rows = sample_rows(p, seed=10 + k)
            xo, fl = oracle.solve_rows(rows, p, i, v, fixed, r.lam, w=ww)
            assert (fl == 0).all()
            rel = np.linalg.norm(xg[rows] - xo, axis=1) / np.linalg.norm(xo, axis=1)
            log(f"  {side}: {rows.size} sampled rows, rel p50={np.median(rel):.2e} max={rel.max():.2e}")
            assert rel.max() <= ROW_TOL
