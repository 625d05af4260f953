"""Pins of the elementwise oracle (SpAdd and the Hadamard product, paper
Section 5.2) against what the definitions fix independently of it: dense
numpy arithmetic on small matrices (brute force), closed forms (A + A = 2A,
A .* A = squares, A + (-A) keeps A's pattern with zeros, disjoint patterns),
and invariance under relabelling rows and columns."""
import numpy as np
import pytest

import matgen
from oracle import elementwise as ew


def dense(M):
    D = np.zeros((M.nrows, M.ncols))
    P = np.zeros((M.nrows, M.ncols), dtype=bool)
    rows = np.repeat(np.arange(M.nrows), np.diff(M.row_ptr))
    D[rows, M.col_idx] = M.val.astype(np.float64)
    P[rows, M.col_idx] = True
    return D, P


def to_dense(R, shape):
    D = np.zeros(shape)
    P = np.zeros(shape, dtype=bool)
    rows = np.repeat(np.arange(shape[0]), np.diff(R.row_ptr))
    D[rows, R.col_idx] = R.val.astype(np.float64)
    P[rows, R.col_idx] = True
    return D, P


def assert_canonical(R, shape):
    rp = R.row_ptr
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0) and rp[-1] == len(R.col_idx)
    for i in range(shape[0]):
        c = R.col_idx[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0) and (len(c) == 0 or (c[0] >= 0 and c[-1] < shape[1]))


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("shape,da,db", [((1, 1), 1.0, 1.0), ((7, 9), 0.3, 0.5), ((40, 33), 0.1, 0.2),
                                         ((16, 64), 0.9, 0.05), ((5, 3), 0.0, 0.6)])
def test_brute_force(shape, da, db, dtype):
    A = matgen.random_sparse(*shape, da, 21, dtype)
    B = matgen.random_sparse(*shape, db, 22, dtype)
    DA, PA = dense(A)
    DB, PB = dense(B)
    S = ew.spadd(A, B)
    assert_canonical(S, shape)
    DS, PS = to_dense(S, shape)
    assert np.array_equal(PS, PA | PB)
    assert np.array_equal(DS, (DA + DB).astype(dtype).astype(np.float64) * PS)
    H = ew.hadamard(A, B)
    assert_canonical(H, shape)
    DH, PH = to_dense(H, shape)
    assert np.array_equal(PH, PA & PB)
    assert np.array_equal(DH, (DA * DB).astype(dtype).astype(np.float64) * PH)


def test_closed_forms():
    A = matgen.rmat(8, 8, seed=23, dtype=np.float64, dist="pm1")
    S = ew.spadd(A, A)
    assert np.array_equal(S.row_ptr, A.row_ptr) and np.array_equal(S.col_idx, A.col_idx)
    assert np.array_equal(S.val, 2 * A.val)
    H = ew.hadamard(A, A)
    assert np.array_equal(H.col_idx, A.col_idx) and np.array_equal(H.val, A.val * A.val)
    N = matgen.CSR(A.nrows, A.ncols, A.row_ptr, A.col_idx, -A.val)
    Z = ew.spadd(A, N)
    assert np.array_equal(Z.col_idx, A.col_idx) and np.all(Z.val == 0)   # structural zeros are kept


def test_disjoint_patterns():
    n = 50
    A = matgen.identity(n)
    B = matgen.CSR(n, n, np.arange(n + 1, dtype=np.int32), ((np.arange(n) + 1) % n).astype(np.int32),
                   np.full(n, 3.0))
    assert ew.hadamard(A, B).nnz == 0
    S = ew.spadd(A, B)
    assert S.nnz == 2 * n
    assert sorted(S.val.tolist()) == [1.0] * n + [3.0] * n


def test_relabelling_commutes():
    A = matgen.rmat(9, 8, seed=24, dtype=np.float32)
    B = matgen.shuffled_copy(A, 25)
    # the shuffled copy is a relabelling: same values, same number of entries, canonical
    assert B.nnz == A.nnz and np.array_equal(np.sort(B.val), np.sort(A.val)) and B.is_canonical()
    S1 = ew.spadd(A, B)
    S2 = ew.spadd(B, A)
    assert np.array_equal(S1.col_idx, S2.col_idx) and np.array_equal(S1.val, S2.val)   # + commutes
    H1 = ew.hadamard(A, B)
    H2 = ew.hadamard(B, A)
    assert np.array_equal(H1.col_idx, H2.col_idx) and np.array_equal(H1.val, H2.val)
    assert S1.nnz == A.nnz + B.nnz - H1.nnz
