"""Full-size parity on all five workloads, in the default launch configuration
the benchmark times.

For every workload:
  * the analysis pass's per-row product counts equal the oracle's, row by row;
  * C.row_ptr and C.col_idx match the oracle digests in
    tests/golden/oracle_summaries.txt (written from the oracle by
    tests/golden/make_golden.py);
  * every row of C is compared with the oracle itself, block by block on the
    host's cores: row lengths and columns bit for bit, values within
    tol * sum_k |A[i,k] B[k,j]| (tol 1e-12 for fp64, 1e-5 for fp32, exact zero
    where that sum is zero). GPU blocks are copied back one at a time, so the
    oracle never holds more than a few blocks of C.
"""
import os
import time

import numpy as np
import pytest

import matgen
import oracle
from gpu_util import check_rows_blockwise, col_blocks_sha256_device, golden, row_ptr_sha256

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

WORKERS = min(16, os.cpu_count() or 1)


def progress(msg: str):
    """Progress lines on stdout and, where a gpurun_out folder exists, in a
    log there (so a long check is visibly alive)."""
    print(msg, flush=True)
    out = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "gpurun_out")
    if os.path.isdir(out):
        with open(os.path.join(out, "fullsize_progress.log"), "a") as f:
            f.write(f"{time.strftime('%H:%M:%S')} {msg}\n")


def run_full(name: str):
    import torch
    from paper_2606_20855_amd import wingspan as ws

    g = golden(name)
    A, B = matgen.config(name)
    progress(f"{name}: m={A.nrows} nnz(A)={A.nnz} nnz(B)={B.nnz} dtype={A.val.dtype}")
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")

    # the analysis pass, row by row
    ref_prods = oracle.row_products(A, B)
    got_prods = ws.row_products(dA, dB).cpu().numpy()
    assert np.array_equal(got_prods, ref_prods), f"{name}: per-row product counts differ"
    progress(f"{name}: per-row product counts equal the oracle's on all {A.nrows} rows")

    C = ws.spgemm(dA, dB)
    torch.cuda.synchronize()
    sym, num = ws.wingspan_last_stats(0), ws.wingspan_last_stats(1)
    progress(f"{name}: symbolic rows {sym['rows']} numeric rows {num['rows']}")
    rp = C.row_ptr.cpu().numpy()
    assert sym["total_products"] == int(ref_prods.sum())
    if g:
        assert sym["total_products"] == g["products"]
        assert int(rp[-1]) == g["nnz_c"]
        assert row_ptr_sha256(rp) == g["row_ptr_sha256"]
        assert col_blocks_sha256_device(rp, C.col_idx) == g["col_blocks_sha256"]
        progress(f"{name}: structure matches the oracle digests")

    def fetch(a: int, b: int):
        return C.col_idx[a:b].cpu().numpy(), C.val[a:b].cpu().numpy()

    res = check_rows_blockwise(A, B, rp, fetch, workers=WORKERS, log=progress)
    assert res["rows"] == A.nrows and res["entries"] == int(rp[-1])
    progress(f"{name}: every row checked: {res['rows']} rows, {res['entries']} entries, {res['products']} "
             f"products in {res['blocks']} blocks on {WORKERS} threads, {res['seconds']:.1f} s; worst "
             f"|d|/M = {res['worst']:.2e}")
    del C
    torch.cuda.empty_cache()
    return num


def test_er1000_full_size():
    run_full("er1000")


def test_laplace512_full_size():
    run_full("laplace512")


def test_er_rect_full_size():
    run_full("er_rect")


def test_rmat18_full_size():
    num = run_full("rmat18")
    assert num["rows"]["dense"] > 0


def test_rmat20_full_size():
    num = run_full("rmat20")
    assert num["rows"]["dense"] > 0
