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


def test_holdout_split_partitions_the_ratings():
    r = workload.make_config(1)
    tp, tc, tv, hu, hi, hv = workload.holdout_split(r.row_ptr, r.col, r.val, 0.1,
                                                    workload.holdout_seed(1), min_keep=3)
    assert tp[-1] + hu.size == r.nnz
    assert 0.08 * r.nnz < hu.size < 0.12 * r.nnz
    assert np.diff(tp).min() >= min(3, int(np.diff(r.row_ptr).min()))
    # the union of the two parts is the original set of triples, with no overlap
    rows = np.repeat(np.arange(r.M), np.diff(tp))
    both = np.concatenate([rows.astype(np.int64) * r.N + tc, hu.astype(np.int64) * r.N + hi])
    orig = np.repeat(np.arange(r.M), np.diff(r.row_ptr)).astype(np.int64) * r.N + r.col
    order = np.argsort(both)
    assert np.array_equal(both[order], np.sort(orig))
    vals = np.concatenate([tv, hv])[order]
    assert np.array_equal(vals, r.val[np.argsort(orig)])
    # held-out triples in CSR order; training columns still strictly increasing per row
    key = hu.astype(np.int64) * r.N + hi
    assert np.all(np.diff(key) > 0)
    for u in range(0, r.M, 97):
        assert np.all(np.diff(tc[tp[u]:tp[u + 1]]) > 0)
    again = workload.holdout_split(r.row_ptr, r.col, r.val, 0.1, workload.holdout_seed(1), 3)
    assert all(np.array_equal(a, b) for a, b in zip(again, (tp, tc, tv, hu, hi, hv)))


def test_holdout_split_keeps_min_ratings_of_light_users():
    ptr = np.array([0, 1, 3, 8], dtype=np.int64)
    col = np.array([0, 0, 1, 0, 1, 2, 3, 4], dtype=np.int32)
    val = np.arange(8, dtype=np.uint8)
    tp, tc, tv, hu, hi, hv = workload.holdout_split(ptr, col, val, 1.0, 1, min_keep=2)
    assert list(np.diff(tp)) == [1, 2, 2]
    assert list(hu) == [2, 2, 2] and list(hi) == [2, 3, 4] and list(hv) == [5, 6, 7]


def test_stored_pairs_are_stored_positions():
    r = workload.make_config(1)
    u, i, v = workload.stored_pairs(r.row_ptr, r.col, r.val, 777, 3)
    assert u.size == 777
    key = u.astype(np.int64) * r.N + i
    assert np.all(np.diff(key) > 0)
    for a, b, c in zip(u[:50], i[:50], v[:50]):
        s, e = r.row_ptr[a], r.row_ptr[a + 1]
        k = s + np.searchsorted(r.col[s:e], b)
        assert r.col[k] == b and r.val[k] == c
