"""The synthetic workload generators produce the structures they promise."""
import numpy as np
import pytest

import matgen


def test_er_exact_distinct_per_row():
    A = matgen.er(500, 300, 10, seed=7)
    assert A.is_canonical()
    assert np.all(np.diff(A.row_ptr) == 10)
    assert A.val.dtype == np.float64 and A.val.min() >= -1 and A.val.max() < 1


def test_er_deterministic():
    a, b = matgen.er(100, 100, 5, 3), matgen.er(100, 100, 5, 3)
    assert np.array_equal(a.col_idx, b.col_idx) and np.array_equal(a.val, b.val)
    c = matgen.er(100, 100, 5, 4)
    assert not np.array_equal(a.col_idx, c.col_idx)


def test_er_rect_shapes():
    A, B = matgen.er_rect(1000, 500, 2000, 8, seed=4)
    assert (A.nrows, A.ncols, B.nrows, B.ncols) == (1000, 500, 500, 2000)
    assert A.is_canonical() and B.is_canonical()
    assert np.all(np.diff(A.row_ptr) == 8) and np.all(np.diff(B.row_ptr) == 8)


def test_laplacian_structure():
    g = 512
    L = matgen.laplacian2d(g)
    assert L.is_canonical()
    assert L.nnz == 5 * g * g - 4 * g == 1_308_672
    rows = np.repeat(np.arange(g * g), np.diff(L.row_ptr))
    diag = rows == L.col_idx
    assert np.all(L.val[diag] == 4) and np.all(L.val[~diag] == -1)
    small = matgen.laplacian2d(6).to_dense()
    assert np.array_equal(small, small.T)


def test_rmat_properties():
    A = matgen.rmat(12, 16, seed=5, dtype=np.float32)
    assert A.is_canonical()
    assert A.nrows == A.ncols == 4096
    assert A.nnz <= 16 * 4096
    # values exactly representable in (0, 1]
    assert A.val.dtype == np.float32 and A.val.min() > 0 and A.val.max() <= 1
    k = np.round((1.0 - A.val.astype(np.float64)) * 2 ** 24)
    assert np.array_equal((1.0 - k * 2.0 ** -24).astype(np.float32), A.val)
    # self-loops are kept
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    assert np.any(rows == A.col_idx)
    # heavy tail: hubs at low indices
    deg = np.diff(A.row_ptr)
    assert deg[0] > 20 * np.median(deg[deg > 0])
    # deterministic per seed
    B = matgen.rmat(12, 16, seed=5, dtype=np.float32)
    assert np.array_equal(A.col_idx, B.col_idx) and np.array_equal(A.val, B.val)


def test_rmat_quadrant_marginals():
    # P(row bit = 1) = c + d = 0.24 and P(col bit = 1) = b + d = 0.24 per level,
    # so the mean row index fraction is 0.24 (before duplicate merging).
    A = matgen.rmat(14, 16, seed=9, dtype=np.float64, dist="pm1")
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    top_bit = (rows >> 13) & 1
    col_top = (A.col_idx >> 13) & 1
    # merging duplicates removes mostly low-index (dense) entries, so allow slack
    assert 0.2 < top_bit.mean() < 0.32 and 0.2 < col_top.mean() < 0.32
    assert A.val.min() >= -1 and A.val.max() < 1


def test_random_sparse_canonical():
    A = matgen.random_sparse(30, 40, 0.3, 1, empty_rows=0.5)
    assert A.is_canonical()
    assert np.sum(np.diff(A.row_ptr) == 0) > 0


@pytest.mark.slow
def test_config_sizes():
    A, B = matgen.config("rmat18")
    assert A is B and A.nrows == 262_144 and A.val.dtype == np.float32
    assert 3_900_000 < A.nnz < 4_000_000
    A, B = matgen.config("er_rect")
    assert A.nnz == 8_000_000 and B.nnz == 4_000_000
