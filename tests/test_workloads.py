"""The seeded generators: shapes, nonzero targets, CSR validity and reproducibility."""

import numpy as np
import pytest

from workloads import gen


def _check_csr(m, n, row_ptr, col, val):
    assert row_ptr.dtype == np.int64 and col.dtype == np.int32 and val.dtype == np.float32
    assert row_ptr.shape == (m + 1,) and row_ptr[0] == 0 and row_ptr[-1] == col.size == val.size
    assert np.all(np.diff(row_ptr) >= 0)
    assert np.all(val > 0) and np.all(np.isfinite(val))
    assert col.min() >= 0 and col.max() < n
    rows = np.repeat(np.arange(m), np.diff(row_ptr))
    key = rows.astype(np.int64) * n + col
    assert np.all(np.diff(key) > 0)


def test_config1_planted():
    p = gen.config(1)
    assert (p.m, p.n, p.r, p.nnz) == (1000, 1000, 8, 50_000)
    _check_csr(p.m, p.n, p.row_ptr, p.col, p.val)
    assert p.W0.shape == (1000, 8) and p.H0.shape == (8, 1000)
    assert np.all(p.W0 > 0) and np.all(p.H0 < 0)
    L = p.W0.astype(np.float64) @ p.H0
    assert abs(L.mean() + p.val.mean()) < 0.05 * p.val.mean()
    q = gen.config(1)
    assert np.array_equal(p.col, q.col) and np.array_equal(p.val, q.val)
    assert np.array_equal(p.W0, q.W0)


def test_planted_two_pass_selection_matches_direct():
    g = np.random.default_rng(0)
    W = g.standard_normal((700, 5)).astype(np.float32)
    H = g.standard_normal((5, 600)).astype(np.float32)
    k = 4200
    k1, v1, t1 = gen._top_k_threshold(W, H, k, 3, 97)
    k2, v2, t2 = gen._top_k_threshold(W, H, k, 3, 97, direct_limit=0)
    assert t1 == t2
    o1, o2 = np.argsort(k1), np.argsort(k2)
    assert np.array_equal(k1[o1], k2[o2]) and np.array_equal(v1[o1], v2[o2])


def test_config2_identity():
    p = gen.config(2)
    assert (p.m, p.n, p.r, p.nnz) == (4096, 4096, 3, 4096)
    _check_csr(p.m, p.n, p.row_ptr, p.col, p.val)
    assert np.all(p.val == 1)
    assert abs(p.W0.std() - 0.1) < 0.01


def test_graph_generator_small():
    n, nnz = 20000, 400_000
    row_ptr, col, val = gen.graph_powerlaw(n, nnz, 4)
    _check_csr(n, n, row_ptr, col, val)
    assert nnz <= col.size <= nnz + 2 * n
    assert np.all(np.diff(row_ptr) > 0)
    assert np.all(np.bincount(col, minlength=n) > 0)
    assert np.all(val == np.rint(val)) and val.min() >= 1
    deg = np.diff(row_ptr)
    assert deg.max() > 20 * deg.mean()  # heavy tail


def test_cooccurrence_generator_small():
    m, n, nnz = 20000, 3000, 600_000
    row_ptr, col, val, meta = gen.cooccurrence_zipf(m, n, nnz, 5)
    _check_csr(m, n, row_ptr, col, val)
    assert abs(col.size - nnz) < 0.03 * nnz
    deg = np.diff(row_ptr)
    assert deg[0] == n or deg[0] > 0.95 * n  # the most frequent token co-occurs with almost all
    assert deg[:100].mean() > deg[-1000:].mean()
    assert np.allclose(val, np.log1p(np.rint(np.expm1(val.astype(np.float64)))), atol=1e-6)


@pytest.mark.parametrize("m,n", [(1, 1), (17, 3), (50, 80)])
def test_random_sparse(m, n):
    row_ptr, col, val = gen.random_sparse(m, n, 0.3, 1, empty_rows=min(2, m - 1), heavy_row_frac=0.3)
    _check_csr(m, n, row_ptr, col, val)
