"""wingspan_spgemm_noalloc (the entry point that allocates nothing: its scratch
is a static device array of the library) against wingspan_spgemm with a
caller-owned workspace, through the C ABI, on consecutive calls that share the
static scratch: a large product, then smaller ones (so each call starts on the
previous call's leftovers). Structure bit for bit equal to wingspan_spgemm's
and to the oracle's; values within tol * sum |products| of the oracle."""
import numpy as np
import pytest

import matgen
import oracle
from gpu_util import TOL

pytestmark = pytest.mark.gpu


def both(A, B, options=None):
    import torch
    from paper_2606_20855_amd import wingspan as ws

    print(f"noalloc: A {A.nrows}x{A.ncols} nnz={A.nnz} B nnz={B.nnz} {A.val.dtype} options={options}", flush=True)
    ref = oracle.spgemm(A, B)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")
    Ad, Bd, dt = dA.desc(), dB.desc(), dA.dtype_code
    h = torch.cuda.current_stream().cuda_stream
    cap = max(ref.nnz, 1)
    outs = []
    for noalloc in (False, True):
        rp = torch.full((A.nrows + 1,), -7, dtype=torch.int64, device="cuda:0")
        col = torch.full((cap,), -7, dtype=torch.int32, device="cuda:0")
        val = torch.full((cap,), 7.0, dtype=dA.val.dtype, device="cuda:0")
        if noalloc:
            nnz = ws.wingspan_spgemm_noalloc(Ad, Bd, dt, rp.data_ptr(), col.data_ptr(), val.data_ptr(), cap, h,
                                             options)
        else:
            nbytes = ws.wingspan_spgemm_workspace_size(Ad, Bd, dt, options)
            wsb = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda:0")
            nnz = ws.wingspan_spgemm(Ad, Bd, dt, rp.data_ptr(), col.data_ptr(), val.data_ptr(), cap, wsb.data_ptr(),
                                     nbytes, h, options)
        torch.cuda.synchronize()
        assert nnz == ref.nnz
        outs.append((rp.cpu().numpy(), col[:nnz].cpu().numpy(), val[:nnz].cpu().numpy()))
    (rp0, col0, val0), (rp1, col1, val1) = outs
    assert np.array_equal(rp1, rp0) and np.array_equal(rp1, ref.row_ptr)
    assert np.array_equal(col1, col0) and np.array_equal(col1, ref.col_idx)
    tol = TOL[np.dtype(A.val.dtype)]
    for v in (val0, val1):
        err = np.abs(v.astype(np.float64) - ref.val.astype(np.float64))
        assert np.all(err <= tol * ref.mag)
    return ref


def test_noalloc_matches_workspace_entry_on_consecutive_calls():
    big = matgen.rmat(12, 16, seed=31, dtype=np.float32)
    ref = both(big, big)
    assert ref.nnz > 500_000
    small = matgen.er(300, 300, 12, seed=32)
    both(small, small)
    # smaller still, through the tiers the first calls did not use
    tiny = matgen.random_sparse(40, 50, 0.2, 33, np.float64, empty_rows=0.3)
    tiny_b = matgen.random_sparse(50, 30, 0.3, 34, np.float64, empty_rows=0.3)
    both(tiny, tiny_b, dict(force_spill=1, tiny_max=-1))
    both(tiny, tiny_b)


def test_noalloc_empty_product():
    from paper_2606_20855_amd import wingspan as ws
    import torch

    A = matgen.random_sparse(20, 10, 0.0, 35)
    B = matgen.random_sparse(10, 15, 0.5, 36)
    dA, dB = ws.DeviceCSR.from_host(A, "cuda:0"), ws.DeviceCSR.from_host(B, "cuda:0")
    rp = torch.full((21,), -1, dtype=torch.int64, device="cuda:0")
    nnz = ws.wingspan_spgemm_noalloc(dA.desc(), dB.desc(), dA.dtype_code, rp.data_ptr(), 0, 0, 0,
                                     torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert nnz == 0 and np.all(rp.cpu().numpy() == 0)
