"""Test infrastructure only: the CPU oracle for sparse C = A * B.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package. The GPU library never imports, links or calls it, and the two
share no code. The arithmetic lives in ``spgemm_oracle.c`` (plain C, single
threaded, built with gcc ``-O2 -ffp-contract=off``); this module only moves
numpy arrays in and out of it.

Inputs are any objects with ``nrows``, ``ncols``, ``row_ptr`` (int32),
``col_idx`` (int32) and ``val`` (float32 or float64) attributes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spgemm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, F64 = 0, 1
_ERRORS = {
    -1: "bad argument",
    -2: "row_ptr is not a valid prefix sum",
    -3: "column index out of range",
    -4: "columns not strictly increasing within a row",
    -5: "out of host memory",
    -6: "output capacity exceeded",
}


def build(force: bool = True) -> str:
    """Compile the oracle into liboracle.so next to its source."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _bind(path: str):
    """Load an oracle shared library from `path` and declare its signatures."""
    lib = ctypes.CDLL(path)
    p = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_check_csr.argtypes = [i64, i64, i64, p, p]
    lib.oracle_check_csr.restype = ctypes.c_int
    lib.oracle_row_products.argtypes = [p, p, p, p, i64, p]
    lib.oracle_row_products.restype = ctypes.c_int
    lib.oracle_spgemm_rows.argtypes = [i64, p, p, p, p, p, p, ctypes.c_int,
                                       p, i64, p, p, p, p, i64]
    lib.oracle_spgemm_rows.restype = i64
    return lib


def _load():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = _bind(_LIB)
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dt(val: np.ndarray) -> int:
    if val.dtype == np.float32:
        return F32
    if val.dtype == np.float64:
        return F64
    raise TypeError(f"unsupported value dtype {val.dtype}")


def _c(a: np.ndarray, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


@dataclass
class OracleResult:
    """Rows of C (int64 row_ptr over the selected rows), plus per-entry
    magnitude sums M[i,j] = sum_k |A[i,k] B[k,j]| and per-row product counts."""
    row_ptr: np.ndarray
    col_idx: np.ndarray
    val: np.ndarray
    mag: np.ndarray
    products: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])


def check_csr(M) -> int:
    """0 if M is canonical CSR, else a negative code (see _ERRORS)."""
    lib = _load()
    rp, ci = _c(M.row_ptr, np.int32), _c(M.col_idx, np.int32)
    return lib.oracle_check_csr(M.nrows, M.ncols, len(ci), _ptr(rp), _ptr(ci))


def row_products(A, B, rows=None, lib=None) -> np.ndarray:
    """Per-row count of scalar products A[i,k]*B[k,j] formed by Gustavson."""
    lib = lib or _load()
    rows = np.arange(A.nrows, dtype=np.int64) if rows is None else _c(rows, np.int64)
    out = np.zeros(len(rows), dtype=np.int64)
    arp, aci, brp = _c(A.row_ptr, np.int32), _c(A.col_idx, np.int32), _c(B.row_ptr, np.int32)
    lib.oracle_row_products(_ptr(arp), _ptr(aci), _ptr(brp), _ptr(rows), len(rows), _ptr(out))
    return out


def spgemm(A, B, rows=None, with_mag: bool = True, lib=None, capacity: Optional[int] = None) -> OracleResult:
    """C = A * B restricted to `rows` of A (default: all rows, in order).

    `lib` selects another build of the oracle (used by the mutation test).
    Without `capacity` the oracle runs twice (a counting pass sizes the
    output); with it, the output arrays are allocated at that many entries and
    the oracle runs once (an upper bound of nnz is the sum over the rows of
    min(products of the row, B.ncols)); a capacity that is too small raises."""
    if A.ncols != B.nrows:
        raise ValueError("A.ncols != B.nrows")
    if A.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")
    lib = lib or _load()
    dt = _dt(A.val)
    rows = np.arange(A.nrows, dtype=np.int64) if rows is None else _c(rows, np.int64)
    arp, aci, av = _c(A.row_ptr, np.int32), _c(A.col_idx, np.int32), _c(A.val, A.val.dtype)
    brp, bci, bv = _c(B.row_ptr, np.int32), _c(B.col_idx, np.int32), _c(B.val, B.val.dtype)
    rp = np.zeros(len(rows) + 1, dtype=np.int64)
    args = (B.ncols, _ptr(arp), _ptr(aci), _ptr(av), _ptr(brp), _ptr(bci), _ptr(bv), dt,
            _ptr(rows), len(rows))
    if capacity is None:
        nnz = lib.oracle_spgemm_rows(*args, _ptr(rp), None, None, None, 0)
        if nnz < 0:
            raise RuntimeError(f"oracle: {_ERRORS.get(nnz, nnz)}")
        cap = nnz
    else:
        cap = int(capacity)
    col = np.zeros(max(cap, 1), dtype=np.int32)
    val = np.zeros(max(cap, 1), dtype=A.val.dtype)
    mag = np.zeros(max(cap, 1), dtype=np.float64) if with_mag else None
    got = lib.oracle_spgemm_rows(*args, _ptr(rp), _ptr(col), _ptr(val), _ptr(mag), cap)
    if got < 0 or (capacity is None and got != cap):
        raise RuntimeError(f"oracle: {_ERRORS.get(got, got)}")
    nnz = got
    col, val = col[:nnz], val[:nnz]
    if with_mag:
        mag = mag[:nnz]
    prods = row_products(A, B, rows, lib=lib)
    return OracleResult(rp, col, val, mag if with_mag else np.zeros(0), prods)
