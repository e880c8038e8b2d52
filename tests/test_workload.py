"""Seeded input generator: determinism, exact sizes, distinct sorted positions."""
import numpy as np
import pytest

import workload


def _check_csr(ptr, col, val, M, N, nnz):
    assert ptr.dtype == np.int64 and col.dtype == np.int32 and val.dtype == np.uint8
    assert ptr.size == M + 1 and ptr[0] == 0 and ptr[-1] == nnz
    assert (np.diff(ptr) >= 0).all()
    assert col.min() >= 0 and col.max() < N
    rows = np.repeat(np.arange(M), np.diff(ptr))
    key = rows.astype(np.int64) * N + col
    assert (np.diff(key) > 0).all(), "positions must be distinct and sorted within rows"
    assert val.max() <= 100


@pytest.mark.parametrize("k", [1, 2])
def test_small_configs(k):
    a = workload.make_config(k)
    b = workload.make_config(k)
    cfg = workload.CONFIGS[k]
    _check_csr(a.row_ptr, a.col, a.val, cfg["M"], cfg["N"], cfg["nnz"])
    assert np.array_equal(a.row_ptr, b.row_ptr)
    assert np.array_equal(a.col, b.col)
    assert np.array_equal(a.val, b.val)
    st = workload.realised_stats(a)
    assert 45 <= st["ratings"]["mean"] <= 55


def test_config2_degree_recipe():
    r = workload.make_config(2)
    d = np.diff(r.row_ptr)
    assert d.min() >= 5 and d.max() <= 50_000
    items = np.bincount(r.col, minlength=r.N)
    assert items.max() > 20 * np.median(items)  # popularity skew


def test_exact_degrees():
    deg = workload.exact_degrees(np.array([5.0, 1.0, 1.0, 0.1]), 1, 10, 17)
    assert deg.sum() == 17 and deg.min() >= 1 and deg.max() <= 10


def test_sampling_thread_invariant_and_dense_rows(monkeypatch):
    # rows of every density class: sparse (alias), dense (keyed selection), full
    deg = np.array([3, 40, 200, 399, 400, 0, 1])
    w = np.linspace(1.0, 50.0, 400)
    a = workload.make_custom(len(deg), 400, deg, seed=5, item_weights=w)
    b = workload.make_custom(len(deg), 400, deg, seed=5, item_weights=w)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    _check_csr(a[0], a[1], a[2], len(deg), 400, int(deg.sum()))


def test_init_factors():
    U, V = workload.init_factors(100, 50, 7, seed=3)
    assert U.dtype == np.float32 and U.shape == (100, 7) and V.shape == (50, 7)
    assert abs(float(U.std()) - 0.1) < 0.02
    U2, V2 = workload.init_factors(100, 50, 7, seed=3)
    assert np.array_equal(U, U2) and np.array_equal(V, V2)
