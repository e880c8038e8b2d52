"""Python binding of libals, the MI355X ALS half-sweep (C ABI in include/als.h).

Argument marshalling only: every step of the half-sweep runs in the HIP
kernels of ``csrc/``. PyTorch supplies device memory (fp32 tensors on
``cuda:0``) and the current HIP stream. There is no CPU path: if the compiled
library is missing, importing this package raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
# torch first: its bundled HIP runtime (soname libamdhip64.so.7) then satisfies libals.so's
# dependency, so the process holds one HIP runtime. Opened before torch, libals.so would load
# the system's runtime, torch would load its own beside it, and the library would see no device.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libals.so")

ALS_OK, ALS_ERR_INVALID_ARG, ALS_ERR_BAD_MATRIX, ALS_ERR_OUT_OF_MEMORY, ALS_ERR_HIP, \
    ALS_ERR_NOT_SPD = range(6)
ALS_ROWS_USERS, ALS_ROWS_ITEMS = 0, 1
ALS_MODE_USERS, ALS_MODE_ITEMS, ALS_MODE_TIME = 0, 1, 2
_MODES = {"users": ALS_MODE_USERS, "items": ALS_MODE_ITEMS, "bins": ALS_MODE_TIME,
          "time": ALS_MODE_TIME}
_SIDES = {"users": ALS_ROWS_USERS, "items": ALS_ROWS_ITEMS,
          ALS_ROWS_USERS: ALS_ROWS_USERS, ALS_ROWS_ITEMS: ALS_ROWS_ITEMS}

EXPORTS = ("als_create", "als_half_sweep", "als_last_rmse_in", "als_rmse", "als_flagged_rows",
           "als_get_csc",
           "als_plan_stats", "als_set_profiling", "als_get_profile", "als_set_weights",
           "als_set_phase_timing", "als_get_phase_cycles", "als_predict", "als_set_holdout",
           "als_holdout_rmse", "als_pair_rmse_noalloc", "als_set_nw_prior", "als_sample_hyper", "als_gibbs_half_sweep",
           "als_set_time_bins", "als_tensor_half_sweep", "als_tensor_rmse",
           "als_set_time_nw_prior", "als_sample_time_hyper", "als_tensor_gibbs_half_sweep",
           "als_tensor_sample_alpha",
           "als_destroy", "als_status_str", "als_last_error")

PHASES = ("stage", "gather", "solve", "residual", "reduce")


class ALSError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{message} (status {status})")
        self.status = status


class Tuning(ctypes.Structure):
    _fields_ = [("hub_threshold", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64)]


def _load_library(path=LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is not built; run __graft_entry__.build() (hipcc, gfx950) first")
    lib = ctypes.CDLL(path)
    P, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    st = ctypes.c_int
    lib.als_create.argtypes = [ctypes.POINTER(P), i64, i64, i64, P, P, P, i32, P,
                               ctypes.POINTER(Tuning)]
    lib.als_create.restype = st
    lib.als_half_sweep.argtypes = [P, st, P, f32, P, ctypes.POINTER(ctypes.c_double)]
    lib.als_half_sweep.restype = st
    lib.als_last_rmse_in.argtypes = [P, ctypes.POINTER(ctypes.c_double)]
    lib.als_last_rmse_in.restype = st
    lib.als_rmse.argtypes = [P, P, P, ctypes.POINTER(ctypes.c_double)]
    lib.als_rmse.restype = st
    lib.als_flagged_rows.argtypes = [P]
    lib.als_flagged_rows.restype = i64
    lib.als_get_csc.argtypes = [P, P, P, P]
    lib.als_get_csc.restype = st
    lib.als_plan_stats.argtypes = [P, st, P, i32]
    lib.als_plan_stats.restype = st
    lib.als_set_profiling.argtypes = [P, i32]
    lib.als_set_profiling.restype = st
    lib.als_get_profile.argtypes = [P, i32, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    lib.als_get_profile.restype = st
    lib.als_set_weights.argtypes = [P, P]
    lib.als_set_weights.restype = st
    lib.als_set_phase_timing.argtypes = [P, i32]
    lib.als_set_phase_timing.restype = st
    lib.als_get_phase_cycles.argtypes = [P, st, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double)]
    lib.als_get_phase_cycles.restype = st
    lib.als_predict.argtypes = [P, P, P, i64, P, P, P]
    lib.als_predict.restype = st
    lib.als_set_holdout.argtypes = [P, i64, P, P, P]
    lib.als_set_holdout.restype = st
    lib.als_holdout_rmse.argtypes = [P, P, P, ctypes.POINTER(ctypes.c_double)]
    lib.als_holdout_rmse.restype = st
    lib.als_pair_rmse_noalloc.argtypes = [P, P, P, i64, P, P, P, ctypes.POINTER(ctypes.c_double)]
    lib.als_pair_rmse_noalloc.restype = st
    f64 = ctypes.c_double
    lib.als_set_nw_prior.argtypes = [P, st, P, f64, P, f64]
    lib.als_set_nw_prior.restype = st
    lib.als_sample_hyper.argtypes = [P, st, P, P, P, P, P, P, ctypes.POINTER(ctypes.c_int32)]
    lib.als_sample_hyper.restype = st
    lib.als_gibbs_half_sweep.argtypes = [P, st, P, f32, P, P, P, P,
                                         ctypes.POINTER(ctypes.c_double)]
    lib.als_gibbs_half_sweep.restype = st
    lib.als_set_time_bins.argtypes = [P, i32, P]
    lib.als_set_time_bins.restype = st
    lib.als_tensor_half_sweep.argtypes = [P, st, P, P, P, f32, ctypes.POINTER(ctypes.c_double)]
    lib.als_tensor_half_sweep.restype = st
    lib.als_tensor_rmse.argtypes = [P, P, P, P, ctypes.POINTER(ctypes.c_double)]
    lib.als_tensor_rmse.restype = st
    lib.als_set_time_nw_prior.argtypes = [P, P, f64, P, f64]
    lib.als_set_time_nw_prior.restype = st
    lib.als_sample_time_hyper.argtypes = [P, P, P, P, P, P, P, ctypes.POINTER(ctypes.c_int32)]
    lib.als_sample_time_hyper.restype = st
    lib.als_tensor_gibbs_half_sweep.argtypes = [P, st, P, P, P, f32, P, P, P,
                                                ctypes.POINTER(ctypes.c_double)]
    lib.als_tensor_gibbs_half_sweep.restype = st
    lib.als_tensor_sample_alpha.argtypes = [P, P, P, P, f64, f64, ctypes.POINTER(ctypes.c_double)]
    lib.als_tensor_sample_alpha.restype = st
    lib.als_destroy.argtypes = [P]
    lib.als_destroy.restype = None
    lib.als_status_str.argtypes = [st]
    lib.als_status_str.restype = ctypes.c_char_p
    lib.als_last_error.argtypes = [P]
    lib.als_last_error.restype = ctypes.c_char_p
    return lib


lib = _load_library()


def _np_ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dev_ptr(t, D, rows, name):
    import torch

    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous float32")
    if tuple(t.shape) != (rows, D):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {(rows, D)}")
    return ctypes.c_void_p(t.data_ptr())


class ALS:
    """One rating matrix (CSR by user) and one factor width D on the current HIP device."""

    def __init__(self, n_users, n_items, row_ptr, col, val, D, stream=None, tuning=None):
        import torch

        row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int64)
        col = np.ascontiguousarray(col, dtype=np.int32)
        val = np.ascontiguousarray(val, dtype=np.uint8)
        self.M, self.N, self.D = int(n_users), int(n_items), int(D)
        self.nnz = int(col.size)
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        tun = None
        if tuning is not None:
            tun = Tuning(int(tuning.get("hub_threshold", 0)), int(tuning.get("chunk", 0)),
                         int(tuning.get("workspace_bytes", 0)))
        h = ctypes.c_void_p()
        s = lib.als_create(ctypes.byref(h), self.M, self.N, self.nnz, _np_ptr(row_ptr),
                           _np_ptr(col), _np_ptr(val), self.D, ctypes.c_void_p(stream.cuda_stream),
                           ctypes.byref(tun) if tun is not None else None)
        if s != ALS_OK:
            raise ALSError(s, lib.als_last_error(None).decode())
        self._h = h

    def _check(self, s):
        if s != ALS_OK:
            raise ALSError(s, lib.als_last_error(self._h).decode())

    def half_sweep(self, side, fixed, lam, out, rmse=False, allow_flagged=False):
        """Solve the rows of ``side`` ("users" or "items") into ``out`` with ``fixed`` held.

        ``out`` must hold the previous iterate (rows without ratings and flagged rows
        keep it). Returns the RMSE of the new state if ``rmse`` else None."""
        sd = _SIDES[side]
        users = sd == ALS_ROWS_USERS
        n_rows, n_fixed = (self.M, self.N) if users else (self.N, self.M)
        fp = _dev_ptr(fixed, self.D, n_fixed, "fixed")
        op = _dev_ptr(out, self.D, n_rows, "out")
        r = ctypes.c_double(0.0)
        s = lib.als_half_sweep(self._h, sd, fp, float(lam), op, ctypes.byref(r) if rmse else None)
        if s == ALS_ERR_NOT_SPD and allow_flagged:
            return r.value
        self._check(s)
        return r.value if rmse else None

    def rmse_in(self):
        """RMSE of the state that entered the last half-sweep (computed in its gather pass)."""
        r = ctypes.c_double(0.0)
        self._check(lib.als_last_rmse_in(self._h, ctypes.byref(r)))
        return r.value

    def rmse(self, U, V):
        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        r = ctypes.c_double(0.0)
        self._check(lib.als_rmse(self._h, up, vp, ctypes.byref(r)))
        return r.value

    def flagged_rows(self):
        return int(lib.als_flagged_rows(self._h))

    def csc(self):
        col_ptr = np.empty(self.N + 1, dtype=np.int64)
        row_idx = np.empty(max(self.nnz, 1), dtype=np.int32)
        vt = np.empty(max(self.nnz, 1), dtype=np.uint8)
        self._check(lib.als_get_csc(self._h, _np_ptr(col_ptr), _np_ptr(row_idx), _np_ptr(vt)))
        return col_ptr, row_idx[: self.nnz], vt[: self.nnz]

    def plan_stats(self, side):
        out = np.zeros(7, dtype=np.int64)
        self._check(lib.als_plan_stats(self._h, _SIDES[side], _np_ptr(out), 7))
        keys = ("rows_with_ratings", "split_rows", "chunks", "batches", "max_degree",
                "workspace_bytes", "slot_bytes")
        return dict(zip(keys, (int(v) for v in out)))

    def set_profiling(self, on=True, gram_only=False):
        """Per-phase HIP event timing; ``gram_only`` times only the launches that build the
        normal equations (mode 2 of ``als_set_profiling``)."""
        self._check(lib.als_set_profiling(self._h, (2 if gram_only else 1) if on else 0))

    def profile(self):
        res = {}
        for i, name in enumerate(PHASES):
            ms = ctypes.c_double(0.0)
            n = ctypes.c_int64(0)
            self._check(lib.als_get_profile(self._h, i, ctypes.byref(ms), ctypes.byref(n)))
            res[name] = (ms.value, n.value)
        return res

    def set_weights(self, weights):
        """Per-rating weights (CSR order, nnz non-negative floats) for weighted ALS; None
        restores plain ALS."""
        if weights is None:
            self._check(lib.als_set_weights(self._h, None))
            return
        w = np.ascontiguousarray(weights, dtype=np.float32)
        if w.shape != (self.nnz,):
            raise ValueError(f"weights have shape {w.shape}, expected ({self.nnz},)")
        self._check(lib.als_set_weights(self._h, _np_ptr(w)))

    def set_phase_timing(self, on=True):
        """Per-row clocks of the fused row kernel (D > 20); resets the totals."""
        self._check(lib.als_set_phase_timing(self._h, 1 if on else 0))

    def phase_cycles(self, side):
        """(cycles before the factorisation, cycles from it on), summed over rows."""
        g = ctypes.c_double(0.0)
        v = ctypes.c_double(0.0)
        self._check(lib.als_get_phase_cycles(self._h, _SIDES[side], ctypes.byref(g), ctypes.byref(v)))
        return g.value, v.value

    def predict(self, U, V, users, items, out=None):
        """r_hat = u_u . v_i for device int32 tensors ``users`` and ``items`` (one pair per
        element); returns ``out`` (a new fp32 tensor unless given). NaN marks a pair whose
        index is outside the tables."""
        import torch

        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        for t, name in ((users, "users"), (items, "items")):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or \
                    t.dtype != torch.int32 or not t.is_contiguous() or t.dim() != 1:
                raise TypeError(f"{name} must be a contiguous 1-D int32 CUDA tensor")
        n = users.numel()
        if items.numel() != n:
            raise ValueError("users and items differ in length")
        if out is None:
            out = torch.empty(n, dtype=torch.float32, device=users.device)
        elif out.dtype != torch.float32 or not out.is_contiguous() or out.numel() != n or \
                out.device.type != "cuda":
            raise TypeError("out must be a contiguous fp32 CUDA tensor with one element per pair")
        self._check(lib.als_predict(self._h, up, vp, n, ctypes.c_void_p(users.data_ptr()),
                                    ctypes.c_void_p(items.data_ptr()),
                                    ctypes.c_void_p(out.data_ptr())))
        return out

    def set_holdout(self, users, items, ratings):
        """Register held-out (user, item, rating) triples (host arrays) for holdout_rmse."""
        u = np.ascontiguousarray(users, dtype=np.int32)
        i = np.ascontiguousarray(items, dtype=np.int32)
        r = np.ascontiguousarray(ratings, dtype=np.uint8)
        if not (u.shape == i.shape == r.shape) or u.ndim != 1:
            raise ValueError("users, items and ratings must be 1-D arrays of one length")
        self._check(lib.als_set_holdout(self._h, u.size, _np_ptr(u), _np_ptr(i), _np_ptr(r)))

    def holdout_rmse(self, U, V):
        """Validation RMSE of (U, V) on the registered held-out triples."""
        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        r = ctypes.c_double(0.0)
        self._check(lib.als_holdout_rmse(self._h, up, vp, ctypes.byref(r)))
        return r.value

    def pair_rmse_noalloc(self, U, V, users, items, ratings):
        """Validation RMSE of (U, V) on device pairs (contiguous 1-D int32 ``users`` and
        ``items``, uint8 ``ratings`` CUDA tensors) through the allocation-free entry point."""
        import torch

        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        for t, name, dt in ((users, "users", torch.int32), (items, "items", torch.int32),
                            (ratings, "ratings", torch.uint8)):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != dt or \
                    not t.is_contiguous() or t.dim() != 1:
                raise TypeError(f"{name} must be a contiguous 1-D {dt} CUDA tensor")
        n = users.numel()
        if items.numel() != n or ratings.numel() != n:
            raise ValueError("users, items and ratings differ in length")
        r = ctypes.c_double(0.0)
        self._check(lib.als_pair_rmse_noalloc(self._h, up, vp, n,
                                              ctypes.c_void_p(users.data_ptr()),
                                              ctypes.c_void_p(items.data_ptr()),
                                              ctypes.c_void_p(ratings.data_ptr()),
                                              ctypes.byref(r)))
        return r.value

    # ---- Bayesian (BPMF / BPTF) Gibbs step ----------------------------------------------

    def set_nw_prior(self, side, mu0, beta0, W0_inv, nu0):
        """Normal-Wishart hyperprior of one side, or of the time chain with side "time"
        (host arrays)."""
        mu0 = np.ascontiguousarray(mu0, dtype=np.float64)
        W = np.ascontiguousarray(W0_inv, dtype=np.float64)
        if mu0.shape != (self.D,) or W.shape != (self.D, self.D):
            raise ValueError("mu0 must have D entries and W0_inv be D x D")
        if side == "time":
            self._check(lib.als_set_time_nw_prior(self._h, _np_ptr(mu0), float(beta0),
                                                  _np_ptr(W), float(nu0)))
            return
        self._check(lib.als_set_nw_prior(self._h, _SIDES[side], _np_ptr(mu0), float(beta0),
                                         _np_ptr(W), float(nu0)))

    def _hyper_args(self, device, chi2, offdiag, z_mu, mu_out, Lambda_out):
        import torch

        D = self.D
        for t, name, size in ((chi2, "chi2", D), (offdiag, "offdiag", D * (D - 1) // 2),
                              (z_mu, "z_mu", D)):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or \
                    t.dtype != torch.float64 or not t.is_contiguous() or t.numel() != size:
                raise TypeError(f"{name} must be a contiguous fp64 CUDA tensor of {size} values")
        if mu_out is None:
            mu_out = torch.empty(D, dtype=torch.float64, device=device)
        if Lambda_out is None:
            Lambda_out = torch.empty((D, D), dtype=torch.float64, device=device)
        return mu_out, Lambda_out

    def sample_hyper(self, side, X, chi2, offdiag, z_mu, mu_out=None, Lambda_out=None,
                     check=False):
        """Draw (mu, Lambda) of ``side`` given its rows X, or with side "time" those of the
        time chain given T; variates are fp64 CUDA tensors. Returns (mu, Lambda) as fp64
        CUDA tensors."""
        if side == "time":
            tp = _dev_ptr(X, self.D, getattr(self, "n_bins", 0), "T")
        else:
            sd = _SIDES[side]
            n = self.M if sd == ALS_ROWS_USERS else self.N
            xp = _dev_ptr(X, self.D, n, "X")
        mu_out, Lambda_out = self._hyper_args(X.device, chi2, offdiag, z_mu, mu_out, Lambda_out)
        status = ctypes.c_int32(0)
        args = (ctypes.c_void_p(chi2.data_ptr()),
                ctypes.c_void_p(offdiag.data_ptr()) if offdiag.numel() else None,
                ctypes.c_void_p(z_mu.data_ptr()), ctypes.c_void_p(mu_out.data_ptr()),
                ctypes.c_void_p(Lambda_out.data_ptr()), ctypes.byref(status) if check else None)
        if side == "time":
            self._check(lib.als_sample_time_hyper(self._h, tp, *args))
        else:
            self._check(lib.als_sample_hyper(self._h, sd, xp, *args))
        return mu_out, Lambda_out

    def gibbs_half_sweep(self, side, fixed, alpha, Lambda, mu, z, out, rmse=False,
                         allow_flagged=False):
        """Draw every row of ``side`` into ``out`` from its conditional given ``fixed``."""
        import torch

        sd = _SIDES[side]
        users = sd == ALS_ROWS_USERS
        n_rows, n_fixed = (self.M, self.N) if users else (self.N, self.M)
        fp = _dev_ptr(fixed, self.D, n_fixed, "fixed")
        op = _dev_ptr(out, self.D, n_rows, "out")
        zp = _dev_ptr(z, self.D, n_rows, "z")
        for t, name, shape in ((Lambda, "Lambda", (self.D, self.D)), (mu, "mu", (self.D,))):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or \
                    t.dtype != torch.float64 or not t.is_contiguous() or tuple(t.shape) != shape:
                raise TypeError(f"{name} must be a contiguous fp64 CUDA tensor of shape {shape}")
        r = ctypes.c_double(0.0)
        s = lib.als_gibbs_half_sweep(self._h, sd, fp, float(alpha),
                                     ctypes.c_void_p(Lambda.data_ptr()),
                                     ctypes.c_void_p(mu.data_ptr()), zp, op,
                                     ctypes.byref(r) if rmse else None)
        if s == ALS_ERR_NOT_SPD and allow_flagged:
            return r.value
        self._check(s)
        return r.value if rmse else None

    # ---- tensor ALS over time bins ---------------------------------------------------------

    def set_time_bins(self, n_bins, bins):
        """Time bin of every rating (host int array, CSR order), each in [0, n_bins)."""
        b = np.ascontiguousarray(bins, dtype=np.int32)
        if b.shape != (self.nnz,):
            raise ValueError(f"bins have shape {b.shape}, expected ({self.nnz},)")
        self._check(lib.als_set_time_bins(self._h, int(n_bins), _np_ptr(b)))
        self.n_bins = int(n_bins)

    def tensor_half_sweep(self, mode, U, V, T, lam, rmse=False, allow_flagged=False):
        """Solve the rows of ``mode`` ("users", "items" or "bins") in place given the other
        two factors."""
        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        tp = _dev_ptr(T, self.D, getattr(self, "n_bins", 0), "T")
        r = ctypes.c_double(0.0)
        s = lib.als_tensor_half_sweep(self._h, _MODES[mode], up, vp, tp, float(lam),
                                      ctypes.byref(r) if rmse else None)
        if s == ALS_ERR_NOT_SPD and allow_flagged:
            return r.value
        self._check(s)
        return r.value if rmse else None

    def tensor_rmse(self, U, V, T):
        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        tp = _dev_ptr(T, self.D, getattr(self, "n_bins", 0), "T")
        r = ctypes.c_double(0.0)
        self._check(lib.als_tensor_rmse(self._h, up, vp, tp, ctypes.byref(r)))
        return r.value

    # ---- BPTF: the tensor model's Gibbs step -------------------------------------------------

    def tensor_gibbs_half_sweep(self, mode, U, V, T, alpha, Lambda, mu, z, rmse=False,
                                allow_flagged=False):
        """Draw the rows of ``mode`` ("users", "items" or "bins") in place from their
        conditionals given the other two factors; for "bins" (Lambda, mu) are the time
        chain's and the bins are drawn even, then odd."""
        import torch

        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        nb = getattr(self, "n_bins", 0)
        tp = _dev_ptr(T, self.D, nb, "T")
        rows = {ALS_MODE_USERS: self.M, ALS_MODE_ITEMS: self.N, ALS_MODE_TIME: nb}[_MODES[mode]]
        zp = _dev_ptr(z, self.D, rows, "z")
        for t, name, shape in ((Lambda, "Lambda", (self.D, self.D)), (mu, "mu", (self.D,))):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or \
                    t.dtype != torch.float64 or not t.is_contiguous() or tuple(t.shape) != shape:
                raise TypeError(f"{name} must be a contiguous fp64 CUDA tensor of shape {shape}")
        r = ctypes.c_double(0.0)
        s = lib.als_tensor_gibbs_half_sweep(self._h, _MODES[mode], up, vp, tp, float(alpha),
                                            ctypes.c_void_p(Lambda.data_ptr()),
                                            ctypes.c_void_p(mu.data_ptr()), zp,
                                            ctypes.byref(r) if rmse else None)
        if s == ALS_ERR_NOT_SPD and allow_flagged:
            return r.value
        self._check(s)
        return r.value if rmse else None

    def tensor_sample_alpha(self, U, V, T, w0, chi2):
        """Rating precision drawn from its posterior: chi2 / (1 / w0 + sse)."""
        up = _dev_ptr(U, self.D, self.M, "U")
        vp = _dev_ptr(V, self.D, self.N, "V")
        tp = _dev_ptr(T, self.D, getattr(self, "n_bins", 0), "T")
        a = ctypes.c_double(0.0)
        self._check(lib.als_tensor_sample_alpha(self._h, up, vp, tp, float(w0), float(chi2),
                                                ctypes.byref(a)))
        return a.value

    def close(self):
        if getattr(self, "_h", None):
            lib.als_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()
