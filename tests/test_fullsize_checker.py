"""The block-wise checker the full-size GPU tests use, exercised on the CPU:
it accepts a C equal to the oracle's and rejects a wrong row length, a wrong
column and a value outside the tolerance (mistakes planted in copies of the
oracle's own output)."""
import numpy as np
import pytest

import matgen
import oracle
from gpu_util import check_rows_blockwise


@pytest.fixture(scope="module")
def case():
    A = matgen.rmat(10, 16, seed=21, dtype=np.float32)
    ref = oracle.spgemm(A, A)
    return A, ref


def run(A, rp, col, val, block=4000):
    return check_rows_blockwise(A, A, rp, lambda a, b: (col[a:b], val[a:b]), workers=3, block_products=block)


def test_accepts_the_oracle_output(case):
    A, ref = case
    res = run(A, ref.row_ptr, ref.col_idx, ref.val)
    assert res["rows"] == A.nrows and res["entries"] == ref.nnz and res["blocks"] > 3
    assert res["products"] == int(ref.products.sum()) and res["worst"] == 0.0


def test_accepts_a_value_inside_the_tolerance(case):
    A, ref = case
    val = ref.val.copy()
    k = int(np.argmax(ref.mag))
    val[k] = np.float32(ref.val[k] + 0.5e-5 * ref.mag[k])
    res = run(A, ref.row_ptr, ref.col_idx, val)
    assert 0 < res["worst"] <= 1e-5


def test_rejects_a_value_outside_the_tolerance(case):
    A, ref = case
    val = ref.val.copy()
    k = ref.nnz // 2
    val[k] = np.float32(ref.val[k] + 3e-5 * ref.mag[k])
    with pytest.raises(AssertionError, match="outside tolerance"):
        run(A, ref.row_ptr, ref.col_idx, val)


def test_rejects_a_wrong_column(case):
    A, ref = case
    col = ref.col_idx.copy()
    r = int(np.argmax(np.diff(ref.row_ptr)))
    col[ref.row_ptr[r]] += 0 if col[ref.row_ptr[r]] + 1 == col[ref.row_ptr[r] + 1] else 1
    if np.array_equal(col, ref.col_idx):
        col[ref.row_ptr[r] + 1] -= 1
    with pytest.raises(AssertionError, match="col_idx differs"):
        run(A, ref.row_ptr, col, ref.val)


def test_rejects_a_wrong_row_length(case):
    A, ref = case
    rp = ref.row_ptr.copy()
    r = int(np.argmax(np.diff(ref.row_ptr)))
    rp[r + 1] -= 1   # entries of row r and r+1 shift by one
    with pytest.raises(AssertionError, match="entries, the oracle"):
        run(A, rp, ref.col_idx, ref.val)
