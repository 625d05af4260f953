"""Test infrastructure only: the CPU oracle for the elementwise operations of
the paper's sparse linear algebra evaluation (Section 5.2), C = A + B (SpAdd)
and C = A .* B (the Hadamard product), on two CSR matrices of one shape.

These are the plain definitions over the sets of stored coordinates, written
with numpy:
  - the sum is stored on the union of A's and B's coordinates; a coordinate
    stored on one side takes that side's value, one stored on both takes
    a + b, kept even where it is exactly zero (the pattern is structural);
  - the product is stored on the intersection and takes a * b.
Values are formed in double and rounded once to the value type; rows come out
sorted by column. Only the tests, the smoke check and the benchmark may use
this module; the GPU library shares no code with it.
"""
from __future__ import annotations

import numpy as np

from . import OracleResult


def _keys(M) -> np.ndarray:
    """Row-major coordinate keys row * ncols + col of M's stored entries."""
    rp = np.asarray(M.row_ptr, dtype=np.int64)
    rows = np.repeat(np.arange(M.nrows, dtype=np.int64), np.diff(rp))
    return rows * np.int64(max(M.ncols, 1)) + np.asarray(M.col_idx, dtype=np.int64)


def _result(nrows: int, ncols: int, keys: np.ndarray, val: np.ndarray, mag: np.ndarray) -> OracleResult:
    rows = keys // np.int64(max(ncols, 1))
    cols = (keys - rows * np.int64(max(ncols, 1))).astype(np.int32)
    rp = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(np.bincount(rows, minlength=nrows)[:nrows], out=rp[1:])
    return OracleResult(rp, cols, val, mag, np.zeros(nrows, dtype=np.int64))


def _check(A, B):
    if A.nrows != B.nrows or A.ncols != B.ncols:
        raise ValueError("A and B must have the same shape")
    if A.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")


def spadd(A, B) -> OracleResult:
    """C = A + B on the union of the stored coordinates."""
    _check(A, B)
    ka, kb = _keys(A), _keys(B)
    keys = np.concatenate([ka, kb])
    vals = np.concatenate([A.val.astype(np.float64), B.val.astype(np.float64)])
    uniq, inv = np.unique(keys, return_inverse=True)
    s = np.zeros(len(uniq), dtype=np.float64)
    np.add.at(s, inv, vals)      # at most two terms per coordinate: a, or a + b
    m = np.zeros(len(uniq), dtype=np.float64)
    np.add.at(m, inv, np.abs(vals))
    return _result(A.nrows, A.ncols, uniq, s.astype(A.val.dtype), m)


def hadamard(A, B) -> OracleResult:
    """C = A .* B on the intersection of the stored coordinates."""
    _check(A, B)
    ka, kb = _keys(A), _keys(B)
    common, ia, ib = np.intersect1d(ka, kb, assume_unique=True, return_indices=True)
    p = A.val[ia].astype(np.float64) * B.val[ib].astype(np.float64)
    return _result(A.nrows, A.ncols, common, p.astype(A.val.dtype), np.abs(p))
