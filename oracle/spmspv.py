"""Test infrastructure only: the CPU oracle for sparse matrix times sparse
vector, y = A x (SpMSpV, paper Section 5.2), with x given by its sorted
stored indices and their values.

This is the plain definition, row by row from A's CSR arrays: y_i is stored
exactly when row i of A has a stored entry in a column where x is stored
(kept even where the sum is zero: the pattern is structural), and then
y_i = sum over those columns j of A[i, j] * x_j, formed in double in column
order and rounded once to the value type. mag_i = sum |A[i, j] * x_j| bounds
the rounding of any other summation order. Only the tests, the smoke check
and the benchmark may use this module; the GPU library shares no code with it.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class SpVecResult:
    idx: np.ndarray   # int32, strictly increasing
    val: np.ndarray   # value type of A
    mag: np.ndarray   # float64, sum of |products| per stored entry

    @property
    def nnz(self) -> int:
        return int(len(self.idx))


def spmspv(A, x_idx: np.ndarray, x_val: np.ndarray) -> SpVecResult:
    """y = A x for A in CSR (any object with nrows, ncols, row_ptr, col_idx,
    val) and a sparse x of length A.ncols."""
    x_idx = np.asarray(x_idx)
    if x_idx.ndim != 1 or len(x_idx) != len(x_val):
        raise ValueError("x_idx and x_val must be 1-D and of one length")
    if len(x_idx) and (x_idx.min() < 0 or x_idx.max() >= A.ncols or np.any(np.diff(x_idx) <= 0)):
        raise ValueError("x_idx must be strictly increasing in [0, A.ncols)")
    if np.asarray(x_val).dtype != A.val.dtype:
        raise TypeError("x and A must share a value dtype")
    # x as a dense lookup: stored flag and value per column
    stored = np.zeros(A.ncols, dtype=bool)
    xd = np.zeros(A.ncols, dtype=np.float64)
    stored[x_idx] = True
    xd[x_idx] = np.asarray(x_val, dtype=np.float64)
    rp = np.asarray(A.row_ptr, dtype=np.int64)
    rows = np.repeat(np.arange(A.nrows, dtype=np.int64), np.diff(rp))
    hit = stored[A.col_idx]                       # entries meeting a stored x
    prod = A.val[hit].astype(np.float64) * xd[A.col_idx[hit]]
    r = rows[hit]
    y_rows = np.unique(r)
    # sums in column order within each row (entries are column-sorted)
    s = np.zeros(A.nrows, dtype=np.float64)
    m = np.zeros(A.nrows, dtype=np.float64)
    np.add.at(s, r, prod)
    np.add.at(m, r, np.abs(prod))
    return SpVecResult(y_rows.astype(np.int32), s[y_rows].astype(A.val.dtype), m[y_rows])
