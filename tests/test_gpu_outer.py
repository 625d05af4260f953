"""Outer-product SpGEMM (per-workgroup partial Cs merged by a coalesce step)
on the GPU against the oracle's C = A B: the same product as the Gustavson
path, so the structure must match bit for bit and the values within the
tolerance of the sum of |products|."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
import oracle
from gpu_util import assert_matches

pytestmark = pytest.mark.gpu


def run_outer(A, B):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    print(f"outer: A {A.nrows}x{A.ncols} nnz={A.nnz} B {B.nrows}x{B.ncols} nnz={B.nnz} dtype={A.val.dtype}",
          flush=True)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), "cuda:0")
    dB = ws.DeviceCSR.from_host(B, "cuda:0")
    C = ws.spgemm_outer(dAt, dB)
    torch.cuda.synchronize()
    return C.to_host()


def check(A, B, what=""):
    got = run_outer(A, B)
    ref = oracle.spgemm(A, B)
    assert_matches(got, ref, A.val.dtype, what=what)
    return got, ref


@pytest.mark.parametrize("shape", [(0, 0, 0), (0, 5, 3), (4, 0, 6), (5, 6, 0), (1, 1, 1), (3, 2, 7)])
@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_degenerate_shapes(shape, dtype):
    m, k, n = shape
    A = matgen.random_sparse(m, k, 0.7, 71, dtype)
    B = matgen.random_sparse(k, n, 0.7, 72, dtype)
    check(A, B, f"shape {shape}")


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("shape,density", [((60, 70, 80), 0.1), ((200, 150, 300), 0.05), ((33, 1000, 17), 0.2),
                                           ((100, 64, 200), 0.25)])
def test_random(shape, density, dtype):
    # the last shape gives rows of several hundred partial entries: the long-row coalesce
    m, k, n = shape
    A = matgen.random_sparse(m, k, density, 73, dtype, empty_rows=0.2)
    B = matgen.random_sparse(k, n, density, 74, dtype)
    check(A, B, f"random {shape}")


def test_er1000_and_laplacian():
    A, B = matgen.config("er1000")
    got, ref = check(A, B, "er1000")
    assert ref.nnz == got.row_ptr[-1]
    L = matgen.laplacian2d(64)
    got, ref = check(L, L, "laplacian 64")
    # integer-valued products: exact whatever the order
    assert np.array_equal(got.val, ref.val)


def test_rectangular_many_chunks():
    # 64 K products over many workgroups' partial Cs
    A, B = matgen.er_rect(4000, 2000, 4000, 4, 75)
    check(A, B, "er rect")


def test_identity_and_permutation_exact():
    A = matgen.rmat(10, 8, seed=76, dtype=np.float64)
    got = run_outer(matgen.identity(A.nrows), A)
    assert np.array_equal(got.row_ptr, A.row_ptr) and np.array_equal(got.col_idx, A.col_idx)
    assert np.array_equal(got.val, A.val)
    P = matgen.permutation(A.nrows, 77)
    check(P, A, "permutation")


def test_rows_past_the_lds_cap_exact():
    # every row of the arrowhead's square gathers about n partial entries (n > 4096):
    # runs sorted in LDS, one merge pass; integer sums are exact whatever the order
    A = matgen.arrowhead(5000)
    got, ref = check(A, A, "arrowhead 5000")
    assert np.array_equal(got.val, ref.val)
    assert int(np.diff(ref.row_ptr).min()) == A.nrows


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_long_row_of_few_columns(dtype):
    # row 0 of A is full over K = 200000 and B's rows have 3 of 50 columns: row 0 of C
    # gathers ~50 entries from each of ~290 partial Cs, so runs of equal columns span
    # merge tiles and compaction blocks
    K = 200000
    rng = np.random.default_rng(81)
    a_rows = [np.zeros(K, np.int64), np.full(5, 1, np.int64), np.full(3, 2, np.int64)]
    a_cols = [np.arange(K), np.sort(rng.choice(K, 5, replace=False)), np.sort(rng.choice(K, 3, replace=False))]
    rows, cols = np.concatenate(a_rows), np.concatenate(a_cols)
    A = matgen.CSR(3, K, np.array([0, K, K + 5, K + 8], np.int32), cols.astype(np.int32),
                   rng.uniform(-1, 1, len(cols)).astype(dtype))
    assert np.array_equal(np.repeat(np.arange(3), np.diff(A.row_ptr)), rows)
    B = matgen.er(K, 50, 3, 82, dtype)
    got, ref = check(A, B, "one long row")
    assert ref.row_ptr[1] == 50


@pytest.mark.slow
@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_rmat14_square(dtype):
    # heavy-tailed rows: the largest gathers ~165 K partial entries (six merge passes)
    A = matgen.rmat(14, 16, seed=3, dtype=dtype)
    ref_prods = oracle.row_products(A, A)
    assert int(ref_prods.max()) > 100000 and int((ref_prods > 4096).sum()) > 500
    check(A, A, f"rmat14 {np.dtype(dtype).name}")


@pytest.mark.slow
def test_er_rect_full_size():
    """The rectangular Erdos-Renyi product at full size (A 1,000,000 x 500,000
    and B 500,000 x 1,000,000, 8 per row, fp64) through the outer product,
    every row checked against the oracle block by block."""
    import os
    import torch
    from paper_2606_20855_amd import wingspan as ws
    from gpu_util import check_rows_blockwise
    A, B = matgen.config("er_rect")
    print(f"outer er_rect: A {A.nrows}x{A.ncols} B {B.nrows}x{B.ncols}", flush=True)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), "cuda:0")
    dB = ws.DeviceCSR.from_host(B, "cuda:0")
    C = ws.spgemm_outer(dAt, dB)
    torch.cuda.synchronize()
    rp = C.row_ptr.cpu().numpy()
    print(f"outer er_rect: nnz(C) = {int(rp[-1])}", flush=True)

    def fetch(a: int, b: int):
        return C.col_idx[a:b].cpu().numpy(), C.val[a:b].cpu().numpy()

    res = check_rows_blockwise(A, B, rp, fetch, workers=min(16, os.cpu_count() or 1),
                               log=lambda m: print(m, flush=True))
    assert res["rows"] == A.nrows and res["entries"] == int(rp[-1]) and res["products"] == 64_000_000
    print(f"outer er_rect: every row checked, worst |d|/M = {res['worst']:.2e}", flush=True)


def test_capacity_and_workspace_errors():
    import torch
    from paper_2606_20855_amd import wingspan as ws
    A = matgen.er(500, 400, 6, 78)
    B = matgen.er(400, 450, 6, 79)
    ref = oracle.spgemm(A, B)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), "cuda:0")
    dB = ws.DeviceCSR.from_host(B, "cuda:0")
    Atd, Bd = dAt.desc(), dB.desc()
    n0 = ws.wingspan_outer_workspace_size(Atd, Bd, 0)
    w0 = torch.empty(n0, dtype=torch.uint8, device="cuda:0")
    P = ws.wingspan_outer_products(Atd, Bd, w0.data_ptr(), n0)
    assert P == 500 * 6 * 6
    # a workspace that fits the count but not P
    c_rp = torch.empty(501, dtype=torch.int64, device="cuda:0")
    st, _ = ws.wingspan_spgemm_outer(Atd, Bd, ws.F64, c_rp.data_ptr(), 0, 0, 0, w0.data_ptr(), n0, check=False)
    assert ws.STATUS[st] == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"
    nbytes = ws.wingspan_outer_workspace_size(Atd, Bd, P)
    wsb = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    cap = ref.nnz - 1
    c_col = torch.full((cap + 8,), -5, dtype=torch.int32, device="cuda:0")
    c_val = torch.full((cap + 8,), 2.0, dtype=torch.float64, device="cuda:0")
    st, n = ws.wingspan_spgemm_outer(Atd, Bd, ws.F64, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(), cap,
                                     wsb.data_ptr(), nbytes, check=False)
    assert ws.STATUS[st] == "WINGSPAN_ERR_INSUFFICIENT_CAPACITY" and n == ref.nnz
    assert np.array_equal(c_rp.cpu().numpy(), ref.row_ptr)
    assert torch.all(c_col == -5) and torch.all(c_val == 2.0)
    # and with room, the same workspace again
    c_col = torch.empty(ref.nnz, dtype=torch.int32, device="cuda:0")
    c_val = torch.empty(ref.nnz, dtype=torch.float64, device="cuda:0")
    st, n = ws.wingspan_spgemm_outer(Atd, Bd, ws.F64, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(), ref.nnz,
                                     wsb.data_ptr(), nbytes, check=False)
    assert ws.STATUS[st] == "WINGSPAN_OK" and n == ref.nnz
    got = ws.DeviceCSR(500, 450, c_rp, c_col, c_val).to_host()
    assert_matches(got, ref, np.float64, what="after capacity error")
