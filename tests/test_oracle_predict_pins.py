"""Pins of the oracle's held-out prediction and validation RMSE.

A prediction is the dot product of a user's and an item's factor vectors
(Sec. 2.2); the quality measure is the RMSE over validation ratings that
training did not see (Sec. 4.1). Each test fixes a property that does not come
from the oracle itself: hand-derived values, the dense special case (a matrix
product), the training residual pass over the same positions (itself pinned in
test_oracle_pins.py), and exact completion of noise-free low-rank data.
Shapes keep both index ranges inside both factor tables, so a planted index
swap in the oracle gives wrong values rather than an out-of-range read.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _fr(rows):
    return np.array([[float(Fraction(v)) for v in r] for r in rows])


def test_q1_golden_predictions():
    for ex in json.load(open(GOLDEN))["predict"]:
        U, V = _fr(ex["U"]), _fr(ex["V"])
        pred = oracle.predict(ex["users"], ex["items"], U, V)
        want = np.array([float(Fraction(v)) for v in ex["predictions"]])
        assert np.array_equal(pred, want)
        r = np.array(ex["ratings"], dtype=np.float64)
        assert oracle.pair_sse(ex["users"], ex["items"], r, U, V) == float(Fraction(ex["sse"]))
        assert oracle.pair_rmse(ex["users"], ex["items"], r, U, V) ** 2 == pytest.approx(
            float(Fraction(ex["rmse_squared"])), rel=1e-15)


def test_q2_dense_pairs_are_the_matrix_product():
    rng = np.random.default_rng(21)
    n, D = 13, 6
    U = rng.normal(size=(n, D))
    V = rng.normal(size=(n, D))
    uu, ii = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    pred = oracle.predict(uu.ravel(), ii.ravel(), U, V)
    np.testing.assert_allclose(pred.reshape(n, n), U @ V.T, rtol=1e-13, atol=1e-14)


def test_q3_stored_positions_give_the_training_sse():
    from tests.test_oracle_pins import rand_csr

    rng = np.random.default_rng(22)
    M = N = 40
    D = 7
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    U = rng.normal(0, 0.5, size=(M, D))
    V = rng.normal(0, 0.5, size=(N, D))
    users = np.repeat(np.arange(M), np.diff(ptr))
    got = oracle.pair_sse(users, idx, val, U, V)
    assert got == pytest.approx(oracle.sse(ptr, idx, val, U, V), rel=1e-13)


def test_q4_noise_free_low_rank_completion():
    """Rank-k ratings seen on 70 % of the positions determine the rest: after ALS with
    tiny lambda the held-out RMSE vanishes (exact completion)."""
    rng = np.random.default_rng(23)
    M, N, k = 80, 60, 3
    D = k
    Us = rng.normal(size=(M, k))
    Vs = rng.normal(size=(N, k))
    full = (Us @ Vs.T) * 20.0
    ptr = np.arange(M + 1, dtype=np.int64) * N
    col = np.tile(np.arange(N, dtype=np.int32), M)
    rows = np.repeat(np.arange(M), N)
    tp, tc, _, hu, hi, _ = workload.holdout_split(ptr, col, np.zeros(M * N, np.uint8), 0.3,
                                                 seed=5, min_keep=2 * D)
    keep = np.ones(M * N, dtype=bool)
    keep[hu.astype(np.int64) * N + hi] = False
    assert np.array_equal(col[keep], tc)
    tv = full[rows[keep], col[keep]]
    hv = full[hu, hi]
    t = oracle.Trajectory(M, N, tp, tc, tv, rng.normal(0, 0.1, (M, D)), rng.normal(0, 0.1, (N, D)),
                          1e-9)
    before = oracle.pair_rmse(hu, hi, hv, t.U, t.V)
    for _ in range(100):
        t.sweep()
    after = oracle.pair_rmse(hu, hi, hv, t.U, t.V)
    assert before > 0.5 * hv.std()
    assert after / hv.std() < 1e-4


def test_q5_scaling_and_symmetry():
    """r_hat is linear in each of u and v and symmetric under swapping the two sides."""
    rng = np.random.default_rng(24)
    n, D = 17, 5
    U = rng.normal(size=(n, D))
    V = rng.normal(size=(n, D))
    users = rng.integers(0, n, 50)
    items = rng.integers(0, n, 50)
    p = oracle.predict(users, items, U, V)
    # a power-of-two scale is exact in binary floating point, so the equality is bitwise
    assert np.array_equal(oracle.predict(users, items, 4.0 * U, V), 4.0 * p)
    assert np.array_equal(oracle.predict(users, items, U, 0.5 * V), 0.5 * p)
    assert np.array_equal(oracle.predict(items, users, V, U), p)


def test_empty_pairs_and_range_checks():
    U = np.ones((3, 2))
    V = np.ones((4, 2))
    assert oracle.predict([], [], U, V).size == 0
    assert oracle.pair_rmse([], [], [], U, V) == 0.0
    with pytest.raises(ValueError):
        oracle.predict([3], [0], U, V)
    with pytest.raises(ValueError):
        oracle.predict([0], [-1], U, V)
