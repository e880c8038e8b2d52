"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each test fixes one property that the paper's method (Sec. 2.2: alternating
regularised least squares; Sec. 4.1: RMSE over ratings) or plain mathematics
determines, chosen so that a plausible slip in the oracle (a dropped term, a
missing n_s in the regulariser, a transposed operand, a wrong index) breaks at
least one of them.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def rand_csr(rng, M, N, density, rmin=0, rmax=100, real=False, min_deg=0):
    """Random sparsity pattern (each row at least min_deg entries) in CSR."""
    mask = rng.random((M, N)) < density
    for u in range(M):
        if mask[u].sum() < min_deg:
            mask[u, rng.choice(N, size=min_deg, replace=False)] = True
    rows, cols = np.nonzero(mask)
    ptr = np.zeros(M + 1, dtype=np.int64)
    np.add.at(ptr, rows + 1, 1)
    ptr = np.cumsum(ptr)
    if real:
        val = rng.uniform(rmin, rmax, size=rows.size)
    else:
        val = rng.integers(rmin, rmax + 1, size=rows.size).astype(np.float64)
    return ptr, cols.astype(np.int32), val


def dense_of(ptr, idx, val, N):
    M = ptr.size - 1
    A = np.full((M, N), np.nan)
    for s in range(M):
        A[s, idx[ptr[s]:ptr[s + 1]]] = val[ptr[s]:ptr[s + 1]]
    return A


def np_transpose(ptr, idx, val, N):
    """Independent transpose: numpy lexsort on (row, col) keys."""
    M = ptr.size - 1
    rows = np.repeat(np.arange(M), np.diff(ptr))
    order = np.lexsort((rows, idx))
    cptr = np.zeros(N + 1, dtype=np.int64)
    np.add.at(cptr, idx.astype(np.int64) + 1, 1)
    return np.cumsum(cptr), rows[order].astype(np.int32), val[order]


# ---- P0: hand-derived rational worked examples ---------------------------------------------

def test_golden_worked_solves():
    g = json.load(open(GOLDEN))
    for ex in g["solve"]:
        F = np.array([[float(Fraction(v)) for v in row] for row in ex["fixed"]])
        idx = np.array([r[0] for r in ex["ratings"]], dtype=np.int32)
        val = np.array([float(Fraction(r[1])) for r in ex["ratings"]])
        ptr = np.array([0, idx.size], dtype=np.int64)
        lam = float(Fraction(ex["lambda"]))
        X, fl = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((1, ex["D"])))
        want = np.array([float(Fraction(v)) for v in ex["x"]])
        assert fl[0] == 0
        np.testing.assert_allclose(X[0], want, rtol=1e-14, atol=0)


def test_golden_worked_rmse():
    g = json.load(open(GOLDEN))
    for ex in g["rmse"]:
        U = np.array([[float(Fraction(v)) for v in r] for r in ex["U"]])
        V = np.array([[float(Fraction(v)) for v in r] for r in ex["V"]])
        c = ex["csr"]
        ptr = np.array(c["row_ptr"], dtype=np.int64)
        col = np.array(c["col"], dtype=np.int32)
        val = np.array(c["val"], dtype=np.float64)
        assert oracle.sse(ptr, col, val, U, V) == float(Fraction(ex["sse"]))
        assert oracle.rmse(ptr, col, val, U, V) ** 2 == pytest.approx(
            float(Fraction(ex["rmse_squared"])), rel=1e-15)


def _exact_solve(F_int, ratings, lam):
    """Exact rational x = (sum f f^T + lam n I)^{-1} sum r f by Gauss-Jordan elimination."""
    D = len(F_int[0])
    n = len(ratings)
    A = [[Fraction(0)] * D for _ in range(D)]
    b = [Fraction(0)] * D
    for j, r in ratings:
        f = F_int[j]
        for a in range(D):
            b[a] += Fraction(r) * f[a]
            for c in range(D):
                A[a][c] += f[a] * f[c]
    for a in range(D):
        A[a][a] += lam * n
    M = [A[a] + [b[a]] for a in range(D)]
    for c in range(D):
        piv = next(r for r in range(c, D) if M[r][c] != 0)
        M[c], M[piv] = M[piv], M[c]
        for r in range(D):
            if r != c and M[r][c] != 0:
                t = M[r][c] / M[c][c]
                M[r] = [M[r][k] - t * M[c][k] for k in range(D + 1)]
    return [M[a][D] / M[a][a] for a in range(D)]


@pytest.mark.parametrize("D,n", [(1, 1), (2, 3), (3, 5), (4, 4), (5, 12)])
def test_brute_force_rational(D, n):
    """Tiny rows solved exactly in rational arithmetic (dyadic inputs, exact in fp64)."""
    rng = np.random.default_rng(100 + 10 * D + n)
    nf = n + 3
    F_int = [[Fraction(int(v), 8) for v in rng.integers(-16, 17, size=D)] for _ in range(nf)]
    js = rng.choice(nf, size=n, replace=False)
    js.sort()
    ratings = [(int(j), int(rng.integers(0, 101))) for j in js]
    lam = Fraction(1, 16)
    want = np.array([float(v) for v in _exact_solve(F_int, ratings, lam)])
    F = np.array([[float(v) for v in row] for row in F_int])
    ptr = np.array([0, n], dtype=np.int64)
    idx = np.array([j for j, _ in ratings], dtype=np.int32)
    val = np.array([r for _, r in ratings], dtype=np.float64)
    X, fl = oracle.half_sweep(ptr, idx, val, F, float(lam), np.zeros((1, D)))
    assert fl[0] == 0
    np.testing.assert_allclose(X[0], want, rtol=1e-11, atol=1e-12 * np.abs(want).max())


# ---- P1: ridge least squares ------------------------------------------------------------------

@pytest.mark.parametrize("D", [1, 3, 5, 8])
def test_p1_matches_lstsq(D):
    rng = np.random.default_rng(D)
    M, N = 12, 30
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    F = rng.normal(0, 0.7, size=(N, D))
    lam = 0.37
    X, fl = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)))
    assert (fl == 0).all()
    for s in range(M):
        js = idx[ptr[s]:ptr[s + 1]]
        n = js.size
        Aaug = np.vstack([F[js], np.sqrt(lam * n) * np.eye(D)])
        baug = np.concatenate([val[ptr[s]:ptr[s + 1]], np.zeros(D)])
        x_ls = np.linalg.lstsq(Aaug, baug, rcond=None)[0]
        np.testing.assert_allclose(X[s], x_ls, rtol=1e-10, atol=1e-12)


# ---- P2: stationarity of the block objective -------------------------------------------------

def test_p2_gradient_zero():
    rng = np.random.default_rng(2)
    M, N, D, lam = 40, 25, 6, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.4, min_deg=1)
    F = rng.normal(0, 0.1, size=(N, D))
    X, fl = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)))
    for s in range(M):
        js = idx[ptr[s]:ptr[s + 1]]
        r = val[ptr[s]:ptr[s + 1]]
        n = js.size
        # gradient of sum (r - f.x)^2 + lam n |x|^2, straight from the ratings
        resid = F[js] @ X[s] - r
        grad = 2.0 * (F[js].T @ resid + lam * n * X[s])
        b = F[js].T @ r
        assert np.linalg.norm(grad) <= 1e-9 * (np.linalg.norm(b) + 1.0)


# ---- P3: monotone objective ------------------------------------------------------------------

def test_p3_objective_monotone():
    rng = np.random.default_rng(3)
    M, N, D, lam = 60, 45, 5, 0.05
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=2)
    U0 = rng.normal(0, 0.1, size=(M, D))
    V0 = rng.normal(0, 0.1, size=(N, D))
    t = oracle.Trajectory(M, N, ptr, idx, val, U0, V0, lam)
    L = [t.objective()]
    for _ in range(8):
        t.step("items")
        L.append(t.objective())
        t.step("users")
        L.append(t.objective())
    for a, b in zip(L, L[1:]):
        assert b <= a * (1 + 1e-12)
    assert L[-1] < 0.5 * L[0]


# ---- P4: closed forms ------------------------------------------------------------------------

def test_p4_single_rating_sherman_morrison():
    rng = np.random.default_rng(4)
    D, lam = 7, 0.3
    F = rng.normal(size=(5, D))
    for j in range(5):
        r = float(rng.integers(0, 101))
        X, _ = oracle.half_sweep(np.array([0, 1]), np.array([j], dtype=np.int32), np.array([r]), F,
                                 lam, np.zeros((1, D)))
        want = r * F[j] / (F[j] @ F[j] + lam)
        np.testing.assert_allclose(X[0], want, rtol=1e-12)


def test_p4_one_factor():
    rng = np.random.default_rng(5)
    N, lam = 20, 0.11
    F = rng.normal(size=(N, 1))
    ptr, idx, val = rand_csr(rng, 6, N, 0.5, min_deg=1)
    X, _ = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((6, 1)))
    for s in range(6):
        js = idx[ptr[s]:ptr[s + 1]]
        r = val[ptr[s]:ptr[s + 1]]
        want = (r * F[js, 0]).sum() / ((F[js, 0] ** 2).sum() + lam * js.size)
        assert X[s, 0] == pytest.approx(want, rel=1e-13)


def test_p4_orthogonal_rows():
    D, c, lam = 6, 1.5, 0.2
    F = c * np.eye(D)
    r = np.arange(1, D + 1, dtype=np.float64) * 7.0
    X, _ = oracle.half_sweep(np.array([0, D]), np.arange(D, dtype=np.int32), r, F, lam,
                             np.zeros((1, D)))
    np.testing.assert_allclose(X[0], c * r / (c * c + lam * D), rtol=1e-13)


# ---- P5: dense, fully observed case = SVD soft threshold --------------------------------------

def test_p5_dense_soft_threshold():
    rng = np.random.default_rng(6)
    M, N, D = 60, 40, 5
    Uo, _ = np.linalg.qr(rng.normal(size=(M, N)))
    Vo, _ = np.linalg.qr(rng.normal(size=(N, N)))
    sig = np.array([100, 80, 60, 40, 25, 10, 8, 6, 4, 3] + [1.0] * (N - 10))
    A = (Uo[:, :N] * sig) @ Vo.T
    tau = 15.0
    lam = tau / np.sqrt(M * N)
    ptr = np.arange(M + 1, dtype=np.int64) * N
    idx = np.tile(np.arange(N, dtype=np.int32), M)
    val = A.ravel()
    t = oracle.Trajectory(M, N, ptr, idx, val, rng.normal(0, 0.1, (M, D)),
                          rng.normal(0, 0.1, (N, D)), lam)
    for _ in range(400):
        t.sweep()
    s = np.linalg.svd(A, compute_uv=False)
    top = s[:D]
    best = np.where(top > tau, 2 * tau * top - tau * tau, top * top).sum() + (s[D:] ** 2).sum()
    assert t.objective() == pytest.approx(best, rel=1e-8)


# ---- P6: exact low-rank recovery ------------------------------------------------------------

def test_p6_low_rank_recovery():
    rng = np.random.default_rng(7)
    M, N, k = 90, 70, 3
    D = 3
    Us = rng.normal(size=(M, k))
    Vs = rng.normal(size=(N, k))
    mask = rng.random((M, N)) < 0.3
    for u in range(M):
        if mask[u].sum() < 2 * D:
            mask[u, rng.choice(N, 2 * D, replace=False)] = True
    for i in range(N):
        if mask[:, i].sum() < 2 * D:
            mask[rng.choice(M, 2 * D, replace=False), i] = True
    rows, cols = np.nonzero(mask)
    ptr = np.cumsum(np.concatenate([[0], mask.sum(1)])).astype(np.int64)
    val = (Us @ Vs.T)[rows, cols] * 20.0
    t = oracle.Trajectory(M, N, ptr, cols.astype(np.int32), val, rng.normal(0, 0.1, (M, D)),
                          rng.normal(0, 0.1, (N, D)), 1e-9)
    for _ in range(100):
        t.sweep()
    assert t.rmse() / val.std() < 1e-4


# ---- P7: user side on A == item side on A^T --------------------------------------------------

def test_p7_symmetry():
    rng = np.random.default_rng(8)
    M, N, D, lam = 30, 20, 4, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.35, min_deg=1)
    V = rng.normal(0, 0.1, size=(N, D))
    Xu, _ = oracle.half_sweep(ptr, idx, val, V, lam, np.zeros((M, D)))
    # A^T in CSR (items as rows) built independently, then its column view via the oracle
    tptr, tidx, tval = np_transpose(ptr, idx, val, N)
    cptr, cidx, cval = oracle.transpose(tptr, tidx, tval, M)
    Xi, _ = oracle.half_sweep(cptr, cidx, cval, V, lam, np.zeros((M, D)))
    assert np.array_equal(Xu, Xi)


# ---- P8: linearity in the ratings ------------------------------------------------------------

def test_p8_linearity():
    rng = np.random.default_rng(9)
    M, N, D, lam = 25, 18, 5, 0.065
    ptr, idx, v1 = rand_csr(rng, M, N, 0.4, rmax=50, min_deg=1)
    v2 = rng.integers(0, 51, size=v1.size).astype(np.float64)
    F = rng.normal(0, 0.3, size=(N, D))
    z = np.zeros((M, D))
    x1, _ = oracle.half_sweep(ptr, idx, v1, F, lam, z)
    x2, _ = oracle.half_sweep(ptr, idx, v2, F, lam, z)
    x12, _ = oracle.half_sweep(ptr, idx, v1 + v2, F, lam, z)
    x3, _ = oracle.half_sweep(ptr, idx, 3.0 * v1, F, lam, z)
    np.testing.assert_allclose(x12, x1 + x2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(x3, 3.0 * x1, rtol=1e-12, atol=1e-12)


# ---- P9: thread-count invariance -------------------------------------------------------------

def test_p9_thread_invariance():
    rng = np.random.default_rng(10)
    M, N, D, lam = 400, 300, 8, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.05, min_deg=1)
    F = rng.normal(0, 0.1, size=(N, D))
    a, _ = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)), threads=1)
    b, _ = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)), threads=4)
    assert np.array_equal(a, b)
    assert oracle.sse(ptr, idx, val, a, F, threads=1) == oracle.sse(ptr, idx, val, a, F, threads=4)


# ---- P10: transpose against an independent sort-based transpose ------------------------------

def test_p10_transpose():
    rng = np.random.default_rng(11)
    ptr, idx, val = rand_csr(rng, 120, 77, 0.1)
    got = oracle.transpose(ptr, idx, val, 77)
    want = np_transpose(ptr, idx, val, 77)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)


# ---- P11: residual RMSE against the Gram identity (consistency) --------------------------------

def test_p11_rmse_gram_identity():
    rng = np.random.default_rng(12)
    M, N, D = 50, 40, 4
    ptr, idx, val = rand_csr(rng, M, N, 0.3, min_deg=1)
    U = rng.normal(size=(M, D))
    V = rng.normal(size=(N, D))
    tot = 0.0
    for s in range(M):
        js = idx[ptr[s]:ptr[s + 1]]
        r = val[ptr[s]:ptr[s + 1]]
        G = V[js].T @ V[js]
        b = V[js].T @ r
        tot += r @ r - 2 * U[s] @ b + U[s] @ G @ U[s]
    want = np.sqrt(tot / ptr[-1])
    assert oracle.rmse(ptr, idx, val, U, V) == pytest.approx(want, rel=1e-10)


# ---- degenerate cases ------------------------------------------------------------------------

def test_empty_row_unchanged_and_zero_ratings_counted():
    F = np.array([[1.0, 0.0], [0.0, 1.0]])
    ptr = np.array([0, 0, 2], dtype=np.int64)
    idx = np.array([0, 1], dtype=np.int32)
    val = np.array([0.0, 0.0])
    prev = np.array([[3.0, 4.0], [5.0, 6.0]])
    X, fl = oracle.half_sweep(ptr, idx, val, F, 0.5, prev)
    assert fl.tolist() == [2, 0]
    assert X[0].tolist() == [3.0, 4.0]
    # a row whose ratings are all zero is observed and pulled to zero
    assert X[1].tolist() == [0.0, 0.0]


def test_exactly_singular_is_flagged():
    F = np.zeros((3, 2))
    ptr = np.array([0, 2], dtype=np.int64)
    X, fl = oracle.half_sweep(ptr, np.array([0, 2], dtype=np.int32), np.array([5.0, 6.0]), F, 0.0,
                              np.array([[7.0, 8.0]]))
    assert fl[0] == 1
    assert X[0].tolist() == [7.0, 8.0]


def test_nan_fixed_row_is_flagged():
    F = np.array([[1.0, 0.0], [np.nan, 1.0]])
    X, fl = oracle.half_sweep(np.array([0, 2]), np.array([0, 1], dtype=np.int32),
                              np.array([1.0, 2.0]), F, 0.1, np.array([[7.0, 8.0]]))
    assert fl[0] == 1 and X[0].tolist() == [7.0, 8.0]


def test_solve_rows_equals_half_sweep():
    rng = np.random.default_rng(13)
    M, N, D, lam = 70, 50, 6, 0.065
    ptr, idx, val = rand_csr(rng, M, N, 0.2, min_deg=1)
    F = rng.normal(0, 0.1, size=(N, D))
    X, _ = oracle.half_sweep(ptr, idx, val, F, lam, np.zeros((M, D)))
    rows = np.array([0, 5, 69, 33])
    Xs, fl = oracle.solve_rows(rows, ptr, idx, val, F, lam)
    assert np.array_equal(Xs, X[rows])
