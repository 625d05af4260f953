"""A plain host-side CSR container (numpy arrays) used to carry inputs."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class CSR:
    """Compressed sparse rows: the row level is dense, the column level is a
    sorted sparse list, and values sit in a flat element array.

    ``row_ptr`` has ``nrows + 1`` entries with ``row_ptr[0] == 0``; row ``i``
    owns positions ``row_ptr[i] .. row_ptr[i+1]-1`` of ``col_idx`` / ``val``.
    """

    nrows: int
    ncols: int
    row_ptr: np.ndarray
    col_idx: np.ndarray
    val: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1]) if len(self.row_ptr) else 0

    @property
    def dtype(self) -> np.dtype:
        return self.val.dtype

    def astype(self, dtype) -> "CSR":
        return CSR(self.nrows, self.ncols, self.row_ptr, self.col_idx,
                   self.val.astype(dtype))

    def row(self, i: int):
        a, b = int(self.row_ptr[i]), int(self.row_ptr[i + 1])
        return self.col_idx[a:b], self.val[a:b]

    def to_dense(self) -> np.ndarray:
        d = np.zeros((self.nrows, self.ncols), dtype=np.float64)
        rows = np.repeat(np.arange(self.nrows), np.diff(self.row_ptr.astype(np.int64)))
        d[rows, self.col_idx.astype(np.int64)] = self.val
        return d

    def pattern_dense(self) -> np.ndarray:
        d = np.zeros((self.nrows, self.ncols), dtype=np.int64)
        rows = np.repeat(np.arange(self.nrows), np.diff(self.row_ptr.astype(np.int64)))
        d[rows, self.col_idx.astype(np.int64)] = 1
        return d

    def is_canonical(self) -> bool:
        """row_ptr starts at 0, is non-decreasing and ends at nnz; columns lie
        in [0, ncols) and strictly increase within every row."""
        rp = self.row_ptr.astype(np.int64)
        if len(rp) != self.nrows + 1 or rp[0] != 0 or np.any(np.diff(rp) < 0):
            return False
        if rp[-1] != len(self.col_idx) or len(self.val) != len(self.col_idx):
            return False
        c = self.col_idx.astype(np.int64)
        if len(c) and (c.min() < 0 or c.max() >= self.ncols):
            return False
        if len(c) > 1:
            d = np.diff(c)
            # a decrease is only allowed where a new row starts
            starts = np.zeros(len(c), dtype=bool)
            starts[rp[1:-1][rp[1:-1] < len(c)]] = True
            if np.any((d <= 0) & ~starts[1:]):
                return False
        return True
