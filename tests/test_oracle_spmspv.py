"""Pins of the SpMSpV oracle (y = A x with sparse x, paper Section 5.2)
against what the definition fixes independently of it: dense numpy
arithmetic and a boolean product on small inputs (brute force), closed forms
(x = e_j gives column j of A; the identity gives x back; an arrowhead matrix
gives known sums), structural zeros, and invariance under relabelling rows."""
import numpy as np
import pytest

import matgen
from oracle import spmspv as sv


def dense(M):
    D = np.zeros((M.nrows, M.ncols))
    P = np.zeros((M.nrows, M.ncols), dtype=bool)
    rows = np.repeat(np.arange(M.nrows), np.diff(M.row_ptr))
    D[rows, M.col_idx] = M.val.astype(np.float64)
    P[rows, M.col_idx] = True
    return D, P


def dense_vec(n, idx, val):
    d = np.zeros(n)
    p = np.zeros(n, dtype=bool)
    d[idx] = np.asarray(val, dtype=np.float64)
    p[idx] = True
    return d, p


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("shape,da,dx", [((1, 1), 1.0, 1.0), ((7, 9), 0.3, 0.5), ((40, 33), 0.1, 0.2),
                                         ((64, 16), 0.9, 0.1), ((5, 3), 0.0, 0.6), ((30, 50), 0.2, 0.0),
                                         ((0, 4), 0.5, 0.5), ((6, 0), 0.5, 0.5)])
def test_brute_force(shape, da, dx, dtype):
    m, n = shape
    A = matgen.random_sparse(m, n, da, 31, dtype)
    xi, xv = matgen.sparse_vector(n, dx, 32, dtype)
    y = sv.spmspv(A, xi, xv)
    DA, PA = dense(A)
    dxv, px = dense_vec(n, xi, xv)
    pattern = (PA.astype(np.int64) @ px.astype(np.int64)) > 0     # boolean product
    assert np.array_equal(y.idx, np.nonzero(pattern)[0])
    assert y.val.dtype == dtype and y.idx.dtype == np.int32
    ref = DA @ dxv
    mag = np.abs(DA) @ np.abs(dxv)
    assert np.allclose(y.mag, mag[pattern], rtol=1e-12, atol=0)
    tol = (1e-12 if dtype == np.float64 else 1e-6) * mag[pattern] + 1e-300
    assert np.all(np.abs(y.val.astype(np.float64) - ref[pattern]) <= tol)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_unit_vector_gives_column(dtype):
    A = matgen.rmat(9, 8, seed=33, dtype=dtype)
    DA, PA = dense(A)
    for j in (0, 1, 17, A.ncols - 1):
        y = sv.spmspv(A, np.array([j], np.int32), np.array([1.0], dtype))
        assert np.array_equal(y.idx, np.nonzero(PA[:, j])[0])
        assert np.array_equal(y.val, DA[PA[:, j], j].astype(dtype))   # a * 1 is exact


def test_identity_returns_x():
    xi, xv = matgen.sparse_vector(500, 0.1, 34)
    y = sv.spmspv(matgen.identity(500), xi, xv)
    assert np.array_equal(y.idx, xi) and np.array_equal(y.val, xv)


def test_arrowhead_closed_form():
    # ones on the first row, the first column and the diagonal
    n = 300
    A = matgen.arrowhead(n)
    xi, xv = matgen.sparse_vector(n, 0.1, 35, dist="int")
    y = sv.spmspv(A, xi, xv)
    x = np.zeros(n)
    x[xi] = xv
    x0 = 0 in set(xi.tolist())
    # row 0 meets every stored x; row i > 0 meets x_0 and x_i
    expect_idx = np.arange(n) if x0 else np.union1d([0], xi)
    assert np.array_equal(y.idx, expect_idx)
    full = np.where(np.arange(n) == 0, x.sum(), x[0] + x)
    assert np.array_equal(y.val, full[expect_idx])


def test_structural_zeros_kept():
    A = matgen.random_sparse(50, 40, 0.2, 36)
    xi, _ = matgen.sparse_vector(40, 0.3, 37)
    y = sv.spmspv(A, xi, np.zeros(len(xi)))
    _, PA = dense(A)
    px = np.zeros(40, dtype=bool)
    px[xi] = True
    assert np.array_equal(y.idx, np.nonzero(PA[:, px].any(axis=1))[0])
    assert np.all(y.val == 0)


def test_empty_x_and_row_relabelling():
    A = matgen.er(200, 300, 6, 38)
    y = sv.spmspv(A, np.zeros(0, np.int32), np.zeros(0))
    assert y.nnz == 0
    xi, xv = matgen.sparse_vector(300, 0.1, 39)
    y = sv.spmspv(A, xi, xv)
    perm = np.random.default_rng(40).permutation(200)
    # P A: row perm[i] of PA is row i of A
    inv = np.argsort(perm)
    rows = np.repeat(np.arange(200), np.diff(A.row_ptr))
    keys = perm[rows].astype(np.int64) * 300 + A.col_idx
    order = np.argsort(keys)
    rp = np.zeros(201, np.int64)
    np.cumsum(np.bincount(perm[rows], minlength=200), out=rp[1:])
    PA = matgen.CSR(200, 300, rp.astype(np.int32), A.col_idx[order], A.val[order])
    yp = sv.spmspv(PA, xi, xv)
    assert np.array_equal(np.sort(perm[y.idx]), yp.idx)
    got = dict(zip(yp.idx.tolist(), yp.val.tolist()))
    assert all(got[perm[i]] == v for i, v in zip(y.idx.tolist(), y.val.tolist()))
    assert inv is not None


def test_rejects_bad_x():
    A = matgen.random_sparse(5, 6, 0.5, 41)
    with pytest.raises(ValueError):
        sv.spmspv(A, np.array([3, 2], np.int32), np.ones(2))
    with pytest.raises(ValueError):
        sv.spmspv(A, np.array([6], np.int32), np.ones(1))
    with pytest.raises(TypeError):
        sv.spmspv(A, np.array([1], np.int32), np.ones(1, np.float32))


def test_transpose_helper():
    # the GPU path takes A's columns: matgen's transpose must be an exact re-layout
    A = matgen.random_sparse(37, 53, 0.15, 42, np.float32)
    T = matgen.transpose(A)
    DA, PA = dense(A)
    DT, PT = dense(T)
    assert T.nrows == 53 and T.ncols == 37
    assert np.array_equal(PT, PA.T) and np.array_equal(DT, DA.T)
    assert T.val.dtype == np.float32 and T.row_ptr.dtype == np.int32
