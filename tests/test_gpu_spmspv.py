"""SpMSpV (y = A x with sparse x) on the GPU against the oracle. The GPU
takes A's columns (matgen's transpose) and scatters with atomics, so the
summation order varies: indices must match exactly, values within the
tolerance of the sum of |products| (1e-12 relative for double, 1e-5 for
float values, which the GPU accumulates in double and rounds once)."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
from oracle import spmspv as sv

pytestmark = pytest.mark.gpu


def run(A, xi, xv):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    print(f"spmspv: A {A.nrows}x{A.ncols} nnz={A.nnz} nnz(x)={len(xi)} dtype={A.val.dtype}", flush=True)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), "cuda:0")
    x_idx = torch.from_numpy(np.ascontiguousarray(xi, dtype=np.int32)).to("cuda:0")
    x_val = torch.from_numpy(np.ascontiguousarray(xv)).to("cuda:0")
    y_idx, y_val = ws.spmspv(dAt, x_idx, x_val)
    torch.cuda.synchronize()
    return y_idx.cpu().numpy(), y_val.cpu().numpy()


def check(A, xi, xv, what=""):
    gi, gv = run(A, xi, xv)
    ref = sv.spmspv(A, xi, xv)
    assert np.array_equal(gi, ref.idx), f"{what}: indices"
    assert gv.dtype == ref.val.dtype
    rel = 1e-12 if ref.val.dtype == np.float64 else 1e-5
    err = np.abs(gv.astype(np.float64) - ref.val.astype(np.float64))
    bad = err > rel * ref.mag
    assert not bad.any(), f"{what}: {int(bad.sum())} values outside tolerance, first at {ref.idx[bad][:5]}"
    return gi, gv, ref


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("shape,da,dx", [((1, 1), 1.0, 1.0), ((7, 9), 0.3, 0.5), ((40, 33), 0.1, 0.2),
                                         ((64, 16), 0.9, 0.1), ((5, 3), 0.0, 0.6), ((30, 50), 0.2, 0.0),
                                         ((0, 4), 0.5, 0.5), ((6, 0), 0.5, 0.5), ((300, 2000), 0.05, 1.0)])
def test_random(shape, da, dx, dtype):
    m, n = shape
    A = matgen.random_sparse(m, n, da, 51, dtype, empty_rows=0.2)
    xi, xv = matgen.sparse_vector(n, dx, 52, dtype)
    check(A, xi, xv, f"random {shape}")


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_rmat_ten_percent(dtype):
    # the paper's x: 90% sparse; R-MAT columns range from empty to hubs
    A = matgen.rmat(14, 16, seed=53, dtype=dtype, dist="open01" if dtype == np.float32 else "pm1")
    xi, xv = matgen.sparse_vector(A.ncols, 0.1, 54, dtype)
    _, _, ref = check(A, xi, xv, "rmat14")
    assert ref.nnz > 1000


def test_long_column_spans_chunks():
    # the arrowhead's first column has n entries: one x entry's products fill several chunks
    n = 20000
    A = matgen.arrowhead(n)
    xi = np.array([0, 5, 19999], np.int32)
    xv = np.array([0.5, -2.0, 3.0])
    gi, gv, ref = check(A, xi, xv, "arrowhead")
    assert ref.nnz == n


def test_chunk_over_many_short_columns():
    # 200K columns, mostly empty, and x holding half of them: a chunk's products span more x entries than it
    # stages, so it searches the global prefix
    A = matgen.random_sparse(1000, 200_000, 0.00002, 55)
    xi, xv = matgen.sparse_vector(200_000, 0.5, 56)
    check(A, xi, xv, "short columns")


def test_structural_zeros_and_empty_x():
    A = matgen.rmat(10, 8, seed=57, dtype=np.float64)
    xi, _ = matgen.sparse_vector(A.ncols, 0.2, 58)
    gi, gv, ref = check(A, xi, np.zeros(len(xi)), "zero x values")
    assert ref.nnz > 0 and np.all(gv == 0)
    gi, gv, ref = check(A, np.zeros(0, np.int32), np.zeros(0), "empty x")
    assert len(gi) == 0


def test_identity_and_unit_vector_exact():
    xi, xv = matgen.sparse_vector(5000, 0.1, 59)
    gi, gv = run(matgen.identity(5000), xi, xv)
    assert np.array_equal(gi, xi) and np.array_equal(gv, xv)
    A = matgen.er(3000, 2000, 9, 60)
    gi, gv = run(A, np.array([7], np.int32), np.array([1.0]))
    ref = sv.spmspv(A, np.array([7], np.int32), np.array([1.0]))
    assert np.array_equal(gi, ref.idx) and np.array_equal(gv, ref.val)   # one product per entry: exact


def test_capacity_and_invalid_x():
    import torch
    from paper_2606_20855_amd import wingspan as ws
    A = matgen.er(2000, 1500, 8, 61)
    xi, xv = matgen.sparse_vector(1500, 0.1, 62)
    ref = sv.spmspv(A, xi, xv)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), "cuda:0")
    x_idx = torch.from_numpy(xi).to("cuda:0")
    x_val = torch.from_numpy(xv).to("cuda:0")
    nbytes = ws.wingspan_spmspv_workspace_size(dAt.desc(), len(xi))
    wsb = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    cap = ref.nnz // 2
    y_idx = torch.full((cap + 64,), -3, dtype=torch.int32, device="cuda:0")
    y_val = torch.full((cap + 64,), 9.0, dtype=torch.float64, device="cuda:0")
    print(f"spmspv capacity: cap={cap} nnz(y)={ref.nnz}", flush=True)
    st, n = ws.wingspan_spmspv(dAt.desc(), ws.F64, x_idx.data_ptr(), x_val.data_ptr(), len(xi), y_idx.data_ptr(),
                               y_val.data_ptr(), cap, wsb.data_ptr(), nbytes, check=False)
    assert ws.STATUS[st] == "WINGSPAN_ERR_INSUFFICIENT_CAPACITY" and n == ref.nnz
    assert np.array_equal(y_idx[:cap].cpu().numpy(), ref.idx[:cap])
    assert torch.all(y_idx[cap:] == -3) and torch.all(y_val[cap:] == 9.0)
    # out of order, then out of range: rejected before the scatter
    for bad in (np.array([5, 3], np.int32), np.array([3, 1500], np.int32), np.array([-1, 4], np.int32)):
        print(f"spmspv invalid x: {bad.tolist()}", flush=True)
        bi = torch.from_numpy(bad).to("cuda:0")
        bv = torch.ones(2, dtype=torch.float64, device="cuda:0")
        st, _ = ws.wingspan_spmspv(dAt.desc(), ws.F64, bi.data_ptr(), bv.data_ptr(), 2, y_idx.data_ptr(),
                                   y_val.data_ptr(), cap, wsb.data_ptr(), nbytes, check=False)
        assert ws.STATUS[st] == "WINGSPAN_ERR_INVALID_MATRIX"
    # the same workspace after all of that, with room for y
    yi = torch.empty(ref.nnz, dtype=torch.int32, device="cuda:0")
    yv = torch.empty(ref.nnz, dtype=torch.float64, device="cuda:0")
    st, n = ws.wingspan_spmspv(dAt.desc(), ws.F64, x_idx.data_ptr(), x_val.data_ptr(), len(xi), yi.data_ptr(),
                               yv.data_ptr(), ref.nnz, wsb.data_ptr(), nbytes, check=False)
    assert ws.STATUS[st] == "WINGSPAN_OK" and n == ref.nnz
    assert np.array_equal(yi.cpu().numpy(), ref.idx)
    assert np.all(np.abs(yv.cpu().numpy() - ref.val) <= 1e-12 * ref.mag)


def test_rerun_with_new_x():
    A = matgen.rmat(11, 16, seed=63, dtype=np.float32, dist="open01")
    for seed in (64, 65):
        xi, xv = matgen.sparse_vector(A.ncols, 0.1, seed, np.float32)
        check(A, xi, xv, f"x seed {seed}")


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_one_range_over_many_pieces(dtype):
    # y has 3,000 positions (one range of 4096) and 200 K products: the range's sorted products span ~50
    # pieces of 4096, each summing its share in LDS and adding it to y with atomics
    A = matgen.random_sparse(3000, 2000, 0.05, 57, dtype)
    xi, xv = matgen.sparse_vector(2000, 0.7, 58, dtype)
    _, _, ref = check(A, xi, xv, "one range")
    assert int(sv.spmspv(A, xi, xv).nnz) == ref.nnz


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_rmat18_ranges_and_pieces(dtype):
    # 64 ranges of y; R-MAT's low rows gather many products (a range over several pieces) while most ranges
    # sit inside one piece and are written with plain stores
    A = matgen.rmat(18, 8, seed=59, dtype=dtype, dist="open01" if dtype == np.float32 else "pm1")
    xi, xv = matgen.sparse_vector(A.ncols, 0.1, 60, dtype)
    check(A, xi, xv, "rmat18")


def test_wide_y_takes_the_atomic_scatter():
    # y of 9 M positions (more ranges than the bucketed scatter's table takes): the atomic scatter
    rng = np.random.default_rng(61)
    m, n = 9_000_000, 300
    rows = np.sort(rng.choice(m, 20000, replace=False))
    cols = rng.integers(0, n, len(rows))
    order = np.lexsort((cols, rows))
    keys = np.unique(rows[order].astype(np.int64) * n + cols[order])
    r, c = keys // n, keys % n
    rp = np.zeros(m + 1, np.int64)
    np.cumsum(np.bincount(r, minlength=m), out=rp[1:])
    A = matgen.CSR(m, n, rp.astype(np.int32), c.astype(np.int32), rng.uniform(-1, 1, len(c)))
    xi, xv = matgen.sparse_vector(n, 0.5, 62, np.float64)
    check(A, xi, xv, "wide y")
