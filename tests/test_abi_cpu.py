"""The C-ABI library loads and exports every symbol include/als.h declares; host-side
validation of als_create runs before any device work (no GPU needed here)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "als.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(als_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("als_create", "als_half_sweep", "als_rmse", "als_destroy"):
        assert required in names


def test_library_exports_every_declared_symbol():
    import paper_1108_2580_amd as pkg

    lib = ctypes.CDLL(pkg.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in als.h but not exported"
    assert set(pkg.EXPORTS) == set(declared_functions())


def test_status_strings():
    from paper_1108_2580_amd import lib

    for s in range(6):
        assert lib.als_status_str(s)
    assert b"unknown" in lib.als_status_str(99)


def _create(M, N, ptr, col, val, D):
    from paper_1108_2580_amd import lib

    h = ctypes.c_void_p(123)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    st = lib.als_create(ctypes.byref(h), M, N, int(col.size), p(ptr), p(col), p(val), D, None, None)
    return st, h, lib.als_last_error(None).decode()


@pytest.mark.parametrize("case,status", [
    ("unsorted", 2), ("duplicate", 2), ("col_range", 2), ("ptr0", 2), ("ptr_end", 2),
    ("ptr_decreasing", 2), ("D0", 1), ("D129", 1)])
def test_create_validation(case, status):
    ptr = np.array([0, 2, 3], dtype=np.int64)
    col = np.array([0, 2, 1], dtype=np.int32)
    val = np.array([5, 0, 7], dtype=np.uint8)
    D = 4
    if case == "unsorted":
        col = np.array([2, 0, 1], dtype=np.int32)
    elif case == "duplicate":
        col = np.array([1, 1, 1], dtype=np.int32)
    elif case == "col_range":
        col = np.array([0, 3, 1], dtype=np.int32)
    elif case == "ptr0":
        ptr = np.array([1, 2, 3], dtype=np.int64)
    elif case == "ptr_end":
        ptr = np.array([0, 2, 2], dtype=np.int64)
    elif case == "ptr_decreasing":
        ptr = np.array([0, 4, 3], dtype=np.int64)
    elif case == "D0":
        D = 0
    elif case == "D129":
        D = 129
    st, h, msg = _create(2, 3, ptr, col, val, D)
    assert st == status, msg
    assert h.value is None
    assert msg


@pytest.mark.parametrize("case", ["users_2_31", "nnz_2_31", "staged_4GiB", "staged_max_ok_shape",
                                  "negative_tuning"])
def test_create_size_limits(case):
    """The shape limits of als_create are checked on the host before any device call: row
    counts below 2^31, nnz below 2^31, and the staged fixed side (max(M, N) + 1) rows of
    16 * ceil(D / 16) floats below 4 GiB (32-bit gather offsets)."""
    from paper_1108_2580_amd import Tuning, lib

    ptr = np.array([0, 2, 3], dtype=np.int64)
    col = np.array([0, 2, 1], dtype=np.int32)
    val = np.array([5, 0, 7], dtype=np.uint8)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    h = ctypes.c_void_p(123)
    M, N, nnz, D, tun = 2, 3, 3, 4, None
    if case == "users_2_31":
        M = 1 << 31
    elif case == "nnz_2_31":
        nnz = 1 << 31
    elif case == "staged_4GiB":
        # D = 128: 512 bytes per staged row; 2^23 - 1 rows plus the zero row reach 4 GiB
        M, D = (1 << 23) - 1, 128
    elif case == "staged_max_ok_shape":
        # 2^23 - 2 rows (plus the zero row) fit; the call then reaches the CSR checks, and a
        # row_ptr that does not start at 0 stops it there, before any device call
        M, D = (1 << 23) - 2, 128
        ptr = np.ones(M + 1, dtype=np.int64)
    elif case == "negative_tuning":
        tun = Tuning(-1, 0, 0)
    st = lib.als_create(ctypes.byref(h), M, N, nnz, p(ptr), p(col), p(val), D, None,
                        None if tun is None else ctypes.byref(tun))
    msg = lib.als_last_error(None).decode()
    assert h.value is None
    if case == "staged_max_ok_shape":
        assert st == 2 and "row_ptr[0]" in msg, msg
    else:
        assert st == 1, msg
        assert msg
