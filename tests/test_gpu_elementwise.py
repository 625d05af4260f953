"""SpAdd (C = A + B) and the Hadamard product (C = A .* B) on the GPU against
the elementwise oracle. Values are formed in double and rounded once on both
sides, so structure and values must match bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
from oracle import elementwise as ew_oracle

pytestmark = pytest.mark.gpu

OPS = {"add": ew_oracle.spadd, "hadamard": ew_oracle.hadamard}


def run(op, A, B):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    print(f"elementwise {op}: {A.nrows}x{A.ncols} nnz(A)={A.nnz} nnz(B)={B.nnz} dtype={A.val.dtype}", flush=True)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")
    C = ws.elementwise(op, dA, dB)
    torch.cuda.synchronize()
    return C.to_host()


def check(op, A, B, what=""):
    got = run(op, A, B)
    ref = OPS[op](A, B)
    assert np.array_equal(np.asarray(got.row_ptr, np.int64), ref.row_ptr), f"{what}: row_ptr"
    assert np.array_equal(got.col_idx, ref.col_idx), f"{what}: col_idx"
    assert got.val.dtype == ref.val.dtype
    assert np.array_equal(got.val.view(np.uint8), ref.val.view(np.uint8)), f"{what}: values not bit-exact"
    return got, ref


@pytest.mark.parametrize("op", ["add", "hadamard"])
@pytest.mark.parametrize("shape,da,db", [((0, 0), 0.5, 0.5), ((0, 7), 0.5, 0.5), ((6, 0), 0.5, 0.5),
                                         ((1, 1), 1.0, 1.0), ((9, 13), 0.4, 0.0), ((9, 13), 0.0, 0.4),
                                         ((50, 70), 0.1, 0.3), ((300, 200), 0.05, 0.05)])
@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_random(op, shape, da, db, dtype):
    A = matgen.random_sparse(*shape, da, 31, dtype, empty_rows=0.2)
    B = matgen.random_sparse(*shape, db, 32, dtype)
    check(op, A, B, what=f"{op} {shape}")


@pytest.mark.parametrize("op", ["add", "hadamard"])
@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_rmat_identity_and_shuffled(op, dtype):
    # the paper's two cases: A = B, and B a shuffled copy of A
    A = matgen.rmat(12, 16, seed=33, dtype=dtype, dist="open01" if dtype == np.float32 else "pm1")
    got, ref = check(op, A, A, what=f"{op} identity")
    assert ref.nnz == A.nnz
    B = matgen.shuffled_copy(A, 34)
    check(op, A, B, what=f"{op} shuffled")


@pytest.mark.parametrize("op", ["add", "hadamard"])
def test_laplacian_and_rectangular(op):
    L = matgen.laplacian2d(96)
    check(op, L, matgen.shuffled_copy(L, 35), what=f"{op} laplacian")
    R1 = matgen.er(3000, 5000, 8, 37)
    check(op, R1, matgen.er(3000, 5000, 8, 38), what=f"{op} er 3000x5000")


@pytest.mark.parametrize("op", ["add", "hadamard"])
def test_dense_rows(op):
    # full rows of 4096 entries: chunks inside one row
    A = matgen.arrowhead(4096)
    B = matgen.random_sparse(4096, 4096, 0.3, 39)
    check(op, A, B, what=f"{op} dense rows")


@pytest.mark.parametrize("op", ["add", "hadamard"])
def test_common_coordinates_across_tile_boundaries(op):
    # long rows where B stores all of A's coordinates, or every other one: the
    # merged sequence's tiles (2048 entries) would end between the two entries
    # of a common coordinate at nearly every boundary
    A = matgen.random_sparse(40, 30000, 0.4, 45)
    rng = np.random.default_rng(46)
    B = matgen.CSR(A.nrows, A.ncols, A.row_ptr, A.col_idx, rng.uniform(-1, 1, A.nnz))
    check(op, A, B, what=f"{op} same pattern")
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    keep = np.arange(A.nnz) % 2 == 0
    rp = np.zeros(A.nrows + 1, np.int64)
    np.cumsum(np.bincount(rows[keep], minlength=A.nrows), out=rp[1:])
    H = matgen.CSR(A.nrows, A.ncols, rp.astype(np.int32), A.col_idx[keep], A.val[keep] * 3.0)
    check(op, A, H, what=f"{op} half the pattern")
    check(op, H, A, what=f"{op} half the pattern, swapped")


@pytest.mark.parametrize("op", ["add", "hadamard"])
def test_chunks_over_many_empty_rows(op):
    # 200K rows, 95% empty: a chunk of entries spans more rows than it stages (1024)
    # and finds rows in the global row pointer
    A = matgen.random_sparse(200_000, 64, 0.05, 40, empty_rows=0.95)
    B = matgen.random_sparse(200_000, 64, 0.05, 41, empty_rows=0.9)
    check(op, A, B, what=f"{op} sparse rows")


def test_cancellation_keeps_structure():
    A = matgen.rmat(10, 8, seed=42, dtype=np.float64, dist="pm1")
    N = matgen.CSR(A.nrows, A.ncols, A.row_ptr, A.col_idx, -A.val)
    got, _ = check("add", A, N, what="A + (-A)")
    assert np.array_equal(got.col_idx, A.col_idx) and np.all(got.val == 0)


def test_values_rerun_with_new_values():
    import torch
    from paper_2606_20855_amd import wingspan as ws
    A = matgen.rmat(10, 8, seed=43, dtype=np.float32)
    B = matgen.shuffled_copy(A, 44)
    dA, dB = ws.DeviceCSR.from_host(A, "cuda:0"), ws.DeviceCSR.from_host(B, "cuda:0")
    for op, code in (("add", ws.OP_ADD), ("hadamard", ws.OP_HADAMARD)):
        nbytes = ws.wingspan_elementwise_workspace_size(dA.desc(), dB.desc())
        wsb = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
        rp = torch.empty(A.nrows + 1, dtype=torch.int64, device="cuda:0")
        nnz = ws.wingspan_elementwise_structure(code, dA.desc(), dB.desc(), rp.data_ptr(), wsb.data_ptr(), nbytes)
        col = torch.empty(max(nnz, 1), dtype=torch.int32, device="cuda:0")
        val = torch.empty(max(nnz, 1), dtype=torch.float32, device="cuda:0")
        for scale in (1.0, 0.5):
            A2 = matgen.CSR(A.nrows, A.ncols, A.row_ptr, A.col_idx, (A.val * np.float32(scale)).astype(np.float32))
            dA.val.copy_(torch.from_numpy(A2.val))
            ws.wingspan_elementwise_values(code, dA.desc(), dB.desc(), ws.F32, rp.data_ptr(), col.data_ptr(),
                                           val.data_ptr(), wsb.data_ptr(), nbytes)
            torch.cuda.synchronize()
            ref = OPS[op](A2, B)
            assert np.array_equal(col[:nnz].cpu().numpy(), ref.col_idx)
            assert np.array_equal(val[:nnz].cpu().numpy(), ref.val), f"{op} scale {scale}"


def test_values_after_the_workspace_served_another_call():
    # the values call reuses the tiling a structure call left in the workspace only while nothing else has
    # used that workspace: after an SpGEMM (or the other operation's structure) on the same memory it tiles
    # again, and after a values call of another operation it tiles for its own
    import torch
    from paper_2606_20855_amd import wingspan as ws
    A = matgen.rmat(11, 8, seed=47, dtype=np.float64)
    B = matgen.shuffled_copy(A, 48)
    dA, dB = ws.DeviceCSR.from_host(A, "cuda:0"), ws.DeviceCSR.from_host(B, "cuda:0")
    Ad, Bd = dA.desc(), dB.desc()
    need = max(ws.wingspan_elementwise_workspace_size(Ad, Bd), ws.wingspan_spgemm_workspace_size(Ad, Ad, ws.F64))
    wsb = torch.empty(need, dtype=torch.uint8, device="cuda:0")
    refs = {ws.OP_ADD: ew_oracle.spadd(A, B), ws.OP_HADAMARD: ew_oracle.hadamard(A, B)}
    rps = {}
    for code in refs:
        rps[code] = torch.empty(A.nrows + 1, dtype=torch.int64, device="cuda:0")
        assert ws.wingspan_elementwise_structure(code, Ad, Bd, rps[code].data_ptr(), wsb.data_ptr(),
                                                 need) == refs[code].nnz

    def values(code):
        ref = refs[code]
        col = torch.full((max(ref.nnz, 1),), -1, dtype=torch.int32, device="cuda:0")
        val = torch.full((max(ref.nnz, 1),), np.nan, dtype=torch.float64, device="cuda:0")
        ws.wingspan_elementwise_values(code, Ad, Bd, ws.F64, rps[code].data_ptr(), col.data_ptr(), val.data_ptr(),
                                       wsb.data_ptr(), need)
        torch.cuda.synchronize()
        assert np.array_equal(col[:ref.nnz].cpu().numpy(), ref.col_idx)
        assert np.array_equal(val[:ref.nnz].cpu().numpy().view(np.uint8), ref.val.view(np.uint8))

    values(ws.OP_ADD)          # the workspace holds the product's tiling: tiles again
    values(ws.OP_HADAMARD)     # the sum's tiling is there now
    values(ws.OP_HADAMARD)     # its own, kept
    c_rp = torch.empty(A.nrows + 1, dtype=torch.int64, device="cuda:0")
    ws.wingspan_spgemm_symbolic(Ad, Ad, c_rp.data_ptr(), wsb.data_ptr(), need)
    values(ws.OP_HADAMARD)     # overwritten by the SpGEMM
    assert ws.wingspan_elementwise_structure(ws.OP_ADD, Ad, Bd, rps[ws.OP_ADD].data_ptr(), wsb.data_ptr(),
                                             need) == refs[ws.OP_ADD].nnz
    values(ws.OP_ADD)          # kept from the structure call
