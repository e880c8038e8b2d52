"""fp64 CPU oracle of the ALS half-sweep -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. It shares no code with the HIP library
(``paper_1108_2580_amd``) and neither imports the other; the only common
dependency is the seeded input generator in ``workload``.

Method (paper Sec. 2.2): with one side of the factorisation fixed, each row s of
the other side is the regularised least-squares solution
    x_s = (sum_j f_j f_j^T + lambda n_s I)^{-1} sum_j r_sj f_j,
computed in fp64 by Cholesky (the per-update inversion of Sec. 4.1).
Weighted ALS (wALS, named beside ALS in Sec. 2 and Sec. 4 but not defined there):
the functions taking ``w`` (one non-negative weight per stored rating, in the
same order as ``val``) solve x_s = (sum_j c_sj f_j f_j^T + lambda n_s I)^{-1}
sum_j c_sj r_sj f_j; ``w=None`` is plain ALS, and unit weights reproduce it bitwise.
A prediction is u_u . v_i (Sec. 2.2); RMSE (Sec. 4.1) is taken over the stored
ratings (training) or over a list of held-out (user, item, rating) triples
(validation: ``predict``, ``pair_rmse``). One sweep solves the items with the users fixed, then the users with
the items fixed (the order of Sec. 2.2).

Pins (tests/test_oracle_pins.py) tie every function here to something other
than itself: ridge least squares, stationarity, a monotone objective, closed
forms, the SVD soft-threshold optimum of the dense case, exact low-rank
recovery, symmetry, linearity, thread invariance, an independent transpose
and hand-derived rational worked examples.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "als_oracle.c")


# Optimised for any x86-64 host with AVX2 and FMA (the library is built once and runs on
# other hosts), with floating-point contraction off: every product and sum is rounded as
# written, so the results do not depend on the instruction set or the optimisation level.
CFLAGS = ["-O3", "-march=x86-64-v3", "-ffp-contract=off", "-fopenmp"]


def build(verbose: bool = False) -> str:
    """Compile als_oracle.c into liboracle.so (gcc, OpenMP, strict IEEE fp64)."""
    cmd = ["gcc", *CFLAGS, "-shared", "-fPIC", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None


def _configure(lib):
    """Declare the C signatures on a loaded oracle library."""
    P, i64, i32, f64, c_int = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
                               ctypes.c_int)
    lib.orc_transpose.argtypes = [i64, i64, P, P, P, P, P, P]
    lib.orc_transpose.restype = c_int
    lib.orc_normal_equations.argtypes = [i32, i64, P, P, P, P, f64, P, P]
    lib.orc_normal_equations.restype = None
    lib.orc_cholesky_solve.argtypes = [i32, P, P, P, P]
    lib.orc_cholesky_solve.restype = c_int
    lib.orc_half_sweep.argtypes = [i64, P, P, P, P, i32, P, f64, P, P, c_int]
    lib.orc_half_sweep.restype = i64
    lib.orc_solve_rows.argtypes = [i64, P, P, P, P, P, i32, P, f64, P, P, c_int]
    lib.orc_solve_rows.restype = i64
    lib.orc_sse.argtypes = [i64, P, P, P, P, i32, P, P, P, c_int]
    lib.orc_sse.restype = f64
    lib.orc_weighted_norm.argtypes = [i64, P, i32, P]
    lib.orc_weighted_norm.restype = f64
    lib.orc_gibbs_rows.argtypes = [i64, P, P, P, i32, P, f64, P, P, P, P, P, c_int]
    lib.orc_gibbs_rows.restype = i64
    lib.orc_nw_posterior.argtypes = [i64, i32, P, P, f64, P, f64, P, P, P, P]
    lib.orc_nw_posterior.restype = None
    lib.orc_nw_sample.argtypes = [i32, P, f64, P, P, P, P, P, P]
    lib.orc_nw_sample.restype = c_int
    lib.orc_tensor_rows.argtypes = [i64, P, P, P, P, i32, P, P, f64, P, P, c_int]
    lib.orc_tensor_rows.restype = i64
    lib.orc_tensor_sse.argtypes = [i64, P, P, P, P, i32, P, P, P, c_int]
    lib.orc_tensor_sse.restype = f64
    lib.orc_predict.argtypes = [i64, P, P, i32, P, P, P, c_int]
    lib.orc_predict.restype = None
    lib.orc_pair_sse.argtypes = [i64, P, P, P, i32, P, P, c_int]
    lib.orc_pair_sse.restype = f64
    lib.orc_tensor_gibbs_rows.argtypes = [i64, P, P, P, P, i32, P, P, f64, P, P, P, P, P, c_int]
    lib.orc_tensor_gibbs_rows.restype = i64
    lib.orc_time_rows.argtypes = [i64, P, P, P, P, i32, P, P, f64, P, P, P, i32, P, P, c_int]
    lib.orc_time_rows.restype = i64
    lib.orc_time_posterior.argtypes = [i64, i32, P, P, f64, P, f64, P, P, P, P]
    lib.orc_time_posterior.restype = None
    return lib


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    _lib = _configure(ctypes.CDLL(_LIB_PATH))
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def transpose(ptr, idx, val, n_cols):
    """Compressed rows -> compressed columns (rows ascending inside each column)."""
    ptr, idx, val = _i64(ptr), _i32(idx), _f64(val)
    n_rows = ptr.size - 1
    out_ptr = np.empty(n_cols + 1, dtype=np.int64)
    out_idx = np.empty(idx.size, dtype=np.int32)
    out_val = np.empty(idx.size, dtype=np.float64)
    if _load().orc_transpose(n_rows, n_cols, _p(ptr), _p(idx), _p(val), _p(out_ptr), _p(out_idx),
                             _p(out_val)) != 0:
        raise ValueError("column index out of range")
    return out_ptr, out_idx, out_val


def _opt_f64(w, n):
    if w is None:
        return None
    w = _f64(w)
    if w.shape != (n,):
        raise ValueError(f"weights have shape {w.shape}, expected ({n},)")
    return w


def normal_equations(row, ptr, idx, val, F, lam, w=None):
    """(A, b) of one row: A = sum c f f^T + lam n I, b = sum c r f (fp64, rating order;
    c = 1 without weights)."""
    ptr, idx, val, F = _i64(ptr), _i32(idx), _f64(val), _f64(F)
    w = _opt_f64(w, val.size)
    D = F.shape[1]
    s, e = int(ptr[row]), int(ptr[row + 1])
    A = np.empty((D, D))
    b = np.empty(D)
    _load().orc_normal_equations(D, e - s, _p(idx[s:e]), _p(val[s:e]),
                                 None if w is None else _p(w[s:e]), _p(F), float(lam), _p(A),
                                 _p(b))
    return A, b


def cholesky_solve(A, b):
    """x = A^{-1} b by Cholesky; returns None when A is not numerically SPD."""
    A, b = _f64(A), _f64(b)
    D = b.size
    W = np.zeros((D, D))
    x = np.empty(D)
    if _load().orc_cholesky_solve(D, _p(A), _p(b), _p(W), _p(x)) != 0:
        return None
    return x


def half_sweep(ptr, idx, val, F, lam, X_prev, threads=0, w=None):
    """One half-sweep. Returns (X_new, flags) with flags 0 solved / 1 not SPD / 2 empty.

    Rows that are empty or flagged keep their value from X_prev. ``w``: optional
    per-rating weights (weighted ALS)."""
    ptr, idx, val, F = _i64(ptr), _i32(idx), _f64(val), _f64(F)
    w = _opt_f64(w, val.size)
    X = np.array(X_prev, dtype=np.float64, order="C", copy=True)
    n_rows = ptr.size - 1
    D = F.shape[1]
    assert X.shape == (n_rows, D)
    flags = np.empty(n_rows, dtype=np.int8)
    nflag = _load().orc_half_sweep(n_rows, _p(ptr), _p(idx), _p(val), _p(w), D, _p(F),
                                   float(lam), _p(X), _p(flags), int(threads))
    if nflag < 0:
        raise MemoryError("oracle half-sweep: schedule allocation failed")
    return X, flags


def solve_rows(rows, ptr, idx, val, F, lam, threads=0, w=None):
    """The half-sweep update of the listed rows only: (X_sel, flags)."""
    rows, ptr, idx, val, F = _i64(rows), _i64(ptr), _i32(idx), _f64(val), _f64(F)
    w = _opt_f64(w, val.size)
    D = F.shape[1]
    X = np.empty((rows.size, D))
    flags = np.empty(rows.size, dtype=np.int8)
    _load().orc_solve_rows(rows.size, _p(rows), _p(ptr), _p(idx), _p(val), _p(w), D, _p(F),
                           float(lam), _p(X), _p(flags), int(threads))
    return X, flags


def sse(ptr, idx, val, X, F, threads=0, per_row=False, w=None):
    """Sum of squared residuals over the stored ratings of the rows of X (each
    multiplied by its weight when ``w`` is given)."""
    ptr, idx, val, X, F = _i64(ptr), _i32(idx), _f64(val), _f64(X), _f64(F)
    w = _opt_f64(w, val.size)
    n_rows = ptr.size - 1
    rs = np.empty(n_rows) if per_row else None
    tot = _load().orc_sse(n_rows, _p(ptr), _p(idx), _p(val), _p(w), F.shape[1], _p(X), _p(F),
                          _p(rs), int(threads))
    return (tot, rs) if per_row else tot


def rmse(ptr, idx, val, X, F, threads=0):
    nnz = int(ptr[-1])
    return float(np.sqrt(sse(ptr, idx, val, X, F, threads) / nnz)) if nnz else 0.0


def weighted_norm(ptr, X):
    ptr, X = _i64(ptr), _f64(X)
    return _load().orc_weighted_norm(ptr.size - 1, _p(ptr), X.shape[1], _p(X))


def _pairs(users, items, U, V):
    users, items, U, V = _i32(users), _i32(items), _f64(U), _f64(V)
    if users.shape != items.shape or users.ndim != 1:
        raise ValueError("users and items must be 1-D arrays of one length")
    if U.shape[1] != V.shape[1]:
        raise ValueError("U and V have different widths")
    if users.size and (users.min() < 0 or users.max() >= U.shape[0]
                       or items.min() < 0 or items.max() >= V.shape[0]):
        raise ValueError("pair index out of range")
    return users, items, U, V


def predict(users, items, U, V, threads=0):
    """r_hat = u_u . v_i for each (users[p], items[p]) pair (fp64)."""
    users, items, U, V = _pairs(users, items, U, V)
    out = np.empty(users.size)
    _load().orc_predict(users.size, _p(users), _p(items), U.shape[1], _p(U), _p(V), _p(out),
                        int(threads))
    return out


def pair_sse(users, items, r, U, V, threads=0):
    """Sum of (r - u_u . v_i)^2 over the pairs."""
    users, items, U, V = _pairs(users, items, U, V)
    r = _f64(r)
    if r.shape != users.shape:
        raise ValueError("one rating per pair")
    return _load().orc_pair_sse(users.size, _p(users), _p(items), _p(r), U.shape[1], _p(U),
                                _p(V), int(threads))


def pair_rmse(users, items, r, U, V, threads=0):
    """Validation RMSE (Sec. 4.1) over held-out (user, item, rating) triples."""
    n = int(np.asarray(users).size)
    return float(np.sqrt(pair_sse(users, items, r, U, V, threads) / n)) if n else 0.0


def objective(csr, csc, U, V, lam, threads=0, w=None):
    """L(U,V) = sum c (r - u.v)^2 + lam (sum_u n_u ||u||^2 + sum_i n_i ||v_i||^2), with
    c the per-rating weights in CSR order (1 without them)."""
    ptr, col, val = csr
    cptr = csc[0]
    return (sse(ptr, col, val, U, V, threads, w=w)
            + lam * (weighted_norm(ptr, U) + weighted_norm(cptr, V)))


class Trajectory:
    """Free-running fp64 ALS from the given (fp32) initial factors.

    ``step(side)`` performs one half-sweep: side "items" solves V with U fixed,
    side "users" solves U with V fixed."""

    def __init__(self, M, N, row_ptr, col, val, U0, V0, lam, threads=0, w=None):
        self.csr = (_i64(row_ptr), _i32(col), _f64(val))
        self.csc = transpose(self.csr[0], self.csr[1], self.csr[2], N)
        self.w = _opt_f64(w, self.csr[2].size)
        # the weights travel with the ratings: transposing them as the carried values
        self.w_t = None if self.w is None else transpose(self.csr[0], self.csr[1], self.w, N)[2]
        self.U = _f64(U0).copy()
        self.V = _f64(V0).copy()
        self.lam = float(lam)
        self.threads = threads
        self.nflag = 0

    def step(self, side):
        if side == "items":
            self.V, fl = half_sweep(*self.csc, self.U, self.lam, self.V, self.threads, w=self.w_t)
        else:
            self.U, fl = half_sweep(*self.csr, self.V, self.lam, self.U, self.threads, w=self.w)
        self.nflag = int((fl == 1).sum())
        return self

    def sweep(self):
        return self.step("items").step("users")

    def rmse(self):
        return rmse(*self.csr, self.U, self.V, self.threads)

    def objective(self):
        return objective(self.csr, self.csc, self.U, self.V, self.lam, self.threads, w=self.w)


# ---- Bayesian (BPMF / BPTF) Gibbs step -------------------------------------------------------

def gibbs_rows(ptr, idx, val, F, alpha, Lam, mu, z, X_prev, threads=0):
    """Conditional draw of every row: Lambda* = Lambda + alpha sum f f^T,
    x = mu* + L*^{-T} z. Returns (X, flags); flagged rows (not SPD) keep X_prev."""
    ptr, idx, val, F = _i64(ptr), _i32(idx), _f64(val), _f64(F)
    Lam, mu, z = _f64(Lam), _f64(mu), _f64(z)
    n_rows = ptr.size - 1
    D = F.shape[1]
    if Lam.shape != (D, D) or mu.shape != (D,) or z.shape != (n_rows, D):
        raise ValueError("Lambda must be D x D, mu of length D, z n_rows x D")
    X = np.array(X_prev, dtype=np.float64, order="C", copy=True)
    assert X.shape == (n_rows, D)
    flags = np.empty(n_rows, dtype=np.int8)
    _load().orc_gibbs_rows(n_rows, _p(ptr), _p(idx), _p(val), D, _p(F), float(alpha), _p(Lam),
                           _p(mu), _p(z), _p(X), _p(flags), int(threads))
    return X, flags


def nw_posterior(X, mu0, beta0, W0inv, nu0):
    """Normal-Wishart posterior given the rows of X: (mu*, beta*, W*^{-1}, nu*)."""
    X, mu0, W0inv = _f64(X), _f64(mu0), _f64(W0inv)
    n, D = X.shape
    mu_s = np.empty(D)
    Winv = np.empty((D, D))
    b = ctypes.c_double()
    v = ctypes.c_double()
    _load().orc_nw_posterior(n, D, _p(X), _p(mu0), float(beta0), _p(W0inv), float(nu0),
                             _p(mu_s), _p(Winv), ctypes.byref(b), ctypes.byref(v))
    return mu_s, b.value, Winv, v.value


def nw_sample(mu_s, beta_s, Winv_s, chi2, offd, zmu):
    """Bartlett draw of (mu, Lambda) from the Normal-Wishart with the given parameters;
    chi2[i] ~ chi-square(nu* - i), offd: D (D - 1) / 2 standard normals (strict lower
    triangle, row order), zmu: D standard normals. None if a factorisation fails."""
    mu_s, Winv_s, chi2, zmu = _f64(mu_s), _f64(Winv_s), _f64(chi2), _f64(zmu)
    D = mu_s.size
    offd = _f64(offd) if D > 1 else np.zeros(1)
    mu = np.empty(D)
    Lam = np.empty((D, D))
    if _load().orc_nw_sample(D, _p(mu_s), float(beta_s), _p(Winv_s), _p(chi2), _p(offd),
                             _p(zmu), _p(mu), _p(Lam)) != 0:
        return None
    return mu, Lam


# ---- tensor ALS (time bins) -----------------------------------------------------------------

def tensor_rows(ptr, idx1, idx2, val, F1, F2, lam, X_prev, threads=0):
    """One mode's half-sweep of tensor ALS: the ALS update with fixed vectors
    F1[idx1] * F2[idx2] (elementwise). Returns (X, flags)."""
    ptr, idx1, idx2, val = _i64(ptr), _i32(idx1), _i32(idx2), _f64(val)
    F1, F2 = _f64(F1), _f64(F2)
    if F1.shape[1] != F2.shape[1]:
        raise ValueError("F1 and F2 differ in width")
    if idx1.size and (idx1.min() < 0 or idx1.max() >= F1.shape[0] or idx2.min() < 0
                      or idx2.max() >= F2.shape[0]):
        raise ValueError("index out of range")
    X = np.array(X_prev, dtype=np.float64, order="C", copy=True)
    n_rows = ptr.size - 1
    D = F1.shape[1]
    assert X.shape == (n_rows, D)
    flags = np.empty(n_rows, dtype=np.int8)
    _load().orc_tensor_rows(n_rows, _p(ptr), _p(idx1), _p(idx2), _p(val), D, _p(F1), _p(F2),
                            float(lam), _p(X), _p(flags), int(threads))
    return X, flags


def tensor_sse(ptr, idx1, idx2, val, X, F1, F2, threads=0):
    ptr, idx1, idx2, val = _i64(ptr), _i32(idx1), _i32(idx2), _f64(val)
    X, F1, F2 = _f64(X), _f64(F1), _f64(F2)
    return _load().orc_tensor_sse(ptr.size - 1, _p(ptr), _p(idx1), _p(idx2), _p(val), X.shape[1],
                                  _p(X), _p(F1), _p(F2), int(threads))


def _group_by(keys, n_keys, *payload):
    """Stable counting sort of the ratings by key: (ptr, payload arrays reordered)."""
    keys = np.asarray(keys, dtype=np.int64)
    order = np.argsort(keys, kind="stable")
    ptr = np.zeros(n_keys + 1, dtype=np.int64)
    np.add.at(ptr, keys + 1, 1)
    return (np.cumsum(ptr),) + tuple(np.asarray(a)[order] for a in payload)


class TensorTrajectory:
    """Free-running fp64 tensor ALS over (user, item, time bin) ratings; one sweep solves
    the items, then the users, then the time bins (each with the other two fixed)."""

    def __init__(self, M, N, n_bins, row_ptr, col, bins, val, U0, V0, T0, lam, threads=0):
        row_ptr, col, bins, val = _i64(row_ptr), _i32(col), _i32(bins), _f64(val)
        users = np.repeat(np.arange(M, dtype=np.int32), np.diff(row_ptr))
        self.by_user = (row_ptr, col, bins, val)
        ip, iu, ib, iv = _group_by(col, N, users, bins, val)
        self.by_item = (ip, _i32(iu), _i32(ib), iv)
        tp, tu, ti, tv = _group_by(bins, n_bins, users, col, val)
        self.by_bin = (tp, _i32(tu), _i32(ti), tv)
        self.U, self.V, self.T = _f64(U0).copy(), _f64(V0).copy(), _f64(T0).copy()
        self.lam = float(lam)
        self.threads = threads
        self.nnz = int(row_ptr[-1])

    def step(self, mode):
        if mode == "items":
            p, i1, i2, v = self.by_item
            self.V, fl = tensor_rows(p, i1, i2, v, self.U, self.T, self.lam, self.V, self.threads)
        elif mode == "users":
            p, i1, i2, v = self.by_user
            self.U, fl = tensor_rows(p, i1, i2, v, self.V, self.T, self.lam, self.U, self.threads)
        else:
            p, i1, i2, v = self.by_bin
            self.T, fl = tensor_rows(p, i1, i2, v, self.U, self.V, self.lam, self.T, self.threads)
        self.nflag = int((fl == 1).sum())
        return self

    def sweep(self):
        return self.step("items").step("users").step("bins")

    def rmse(self):
        p, i1, i2, v = self.by_user
        return float(np.sqrt(tensor_sse(p, i1, i2, v, self.U, self.V, self.T, self.threads)
                             / self.nnz)) if self.nnz else 0.0


# ---- BPTF: the tensor model's Gibbs step (time factors as a Markov chain) -----------------------

def _tensor_args(ptr, idx1, idx2, val, F1, F2):
    ptr, idx1, idx2, val = _i64(ptr), _i32(idx1), _i32(idx2), _f64(val)
    F1, F2 = _f64(F1), _f64(F2)
    if F1.shape[1] != F2.shape[1]:
        raise ValueError("F1 and F2 differ in width")
    if idx1.size and (idx1.min() < 0 or idx1.max() >= F1.shape[0] or idx2.min() < 0
                      or idx2.max() >= F2.shape[0]):
        raise ValueError("index out of range")
    return ptr, idx1, idx2, val, F1, F2


def tensor_gibbs_rows(ptr, idx1, idx2, val, F1, F2, alpha, Lam, mu, z, X_prev, threads=0):
    """Conditional draw of every user (or item) row of the tensor model: fixed vectors
    F1[idx1] * F2[idx2], prior N(mu, Lambda^{-1}), rating precision alpha.
    Returns (X, flags); flagged rows keep X_prev."""
    ptr, idx1, idx2, val, F1, F2 = _tensor_args(ptr, idx1, idx2, val, F1, F2)
    Lam, mu, z = _f64(Lam), _f64(mu), _f64(z)
    n_rows, D = ptr.size - 1, F1.shape[1]
    if Lam.shape != (D, D) or mu.shape != (D,) or z.shape != (n_rows, D):
        raise ValueError("Lambda must be D x D, mu of length D, z n_rows x D")
    X = np.array(X_prev, dtype=np.float64, order="C", copy=True)
    assert X.shape == (n_rows, D)
    flags = np.empty(n_rows, dtype=np.int8)
    _load().orc_tensor_gibbs_rows(n_rows, _p(ptr), _p(idx1), _p(idx2), _p(val), D, _p(F1),
                                  _p(F2), float(alpha), _p(Lam), _p(mu), _p(z), _p(X),
                                  _p(flags), int(threads))
    return X, flags


def time_rows(ptr, idx1, idx2, val, F1, F2, alpha, Lam_T, mu_T, z, parity, T_prev, threads=0):
    """Conditional draw of the time bins of one parity (0: bins 0, 2, ...; 1: bins 1, 3, ...)
    under the Markov-chain prior, the other bins fixed. Returns (T, flags); bins of the
    other parity and flagged bins keep T_prev (their flags are 0)."""
    ptr, idx1, idx2, val, F1, F2 = _tensor_args(ptr, idx1, idx2, val, F1, F2)
    Lam_T, mu_T, z = _f64(Lam_T), _f64(mu_T), _f64(z)
    K, D = ptr.size - 1, F1.shape[1]
    if K < 1 or Lam_T.shape != (D, D) or mu_T.shape != (D,) or z.shape != (K, D):
        raise ValueError("need K >= 1, Lambda_T D x D, mu_T of length D, z K x D")
    if parity not in (0, 1):
        raise ValueError("parity is 0 or 1")
    T = np.array(T_prev, dtype=np.float64, order="C", copy=True)
    assert T.shape == (K, D)
    flags = np.zeros(K, dtype=np.int8)
    _load().orc_time_rows(K, _p(ptr), _p(idx1), _p(idx2), _p(val), D, _p(F1), _p(F2),
                          float(alpha), _p(Lam_T), _p(mu_T), _p(z), int(parity), _p(T),
                          _p(flags), int(threads))
    return T, flags


def time_posterior(T, mu0, beta0, W0inv, nu0):
    """Normal-Wishart posterior of (mu_T, Lambda_T) given the chain T (K x D):
    (mu*, beta*, W*^{-1}, nu*)."""
    T, mu0, W0inv = _f64(T), _f64(mu0), _f64(W0inv)
    K, D = T.shape
    if K < 1:
        raise ValueError("the chain needs at least one bin")
    mu_s = np.empty(D)
    Winv = np.empty((D, D))
    b = ctypes.c_double()
    v = ctypes.c_double()
    _load().orc_time_posterior(K, D, _p(T), _p(mu0), float(beta0), _p(W0inv), float(nu0),
                               _p(mu_s), _p(Winv), ctypes.byref(b), ctypes.byref(v))
    return mu_s, b.value, Winv, v.value


def alpha_posterior(sse, n, w0, nu0):
    """Posterior of the rating precision alpha under its one-dimensional Wishart prior
    W(w0, nu0) given the n residuals with sum of squares sse: W(w*, nu*) with
    1 / w* = 1 / w0 + sse and nu* = nu0 + n. A draw is w* times a chi-square(nu*) variate."""
    return 1.0 / (1.0 / float(w0) + float(sse)), float(nu0) + float(n)
