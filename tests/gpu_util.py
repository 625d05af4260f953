"""Helpers for the GPU parity tests: run the library through the C ABI and
compare its output with the CPU oracle."""
from __future__ import annotations

import hashlib
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_golden  # noqa: E402

TOL = {np.dtype(np.float64): 1e-12, np.dtype(np.float32): 1e-5}


def golden(name: str) -> dict:
    return make_golden.read().get(name, {})


def run_gpu(A, B, options=None):
    """C = A * B on cuda:0 through the C ABI; returns (host C, symbolic stats, numeric stats)."""
    import torch
    from paper_2606_20855_amd import wingspan as ws

    print(f"run_gpu: A {A.nrows}x{A.ncols} nnz={A.nnz} B {B.nrows}x{B.ncols} nnz={B.nnz} "
          f"dtype={A.val.dtype} options={options}", flush=True)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")
    C = ws.spgemm(dA, dB, options=options)
    sym = ws.wingspan_last_stats(0)
    num = ws.wingspan_last_stats(1)
    torch.cuda.synchronize()
    return C.to_host(), sym, num


def assert_matches(got, ref, dtype, rows=None, what=""):
    """Structure bit-exact; values within tol * sum |products| (exact zero
    when the magnitude sum is zero)."""
    rp = np.asarray(got.row_ptr, dtype=np.int64)
    if rows is None:
        assert np.array_equal(rp, ref.row_ptr), f"{what}: row_ptr differs"
        col, val = got.col_idx, got.val
    else:
        segs = [(rp[i], rp[i + 1]) for i in rows]
        lens = np.array([b - a for a, b in segs], dtype=np.int64)
        assert np.array_equal(lens, np.diff(ref.row_ptr)), f"{what}: row lengths differ"
        col = np.concatenate([got.col_idx[a:b] for a, b in segs]) if segs else np.zeros(0, np.int32)
        val = np.concatenate([got.val[a:b] for a, b in segs]) if segs else np.zeros(0, dtype)
    assert np.array_equal(col, ref.col_idx), f"{what}: col_idx differs"
    tol = TOL[np.dtype(dtype)]
    err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
    bound = tol * ref.mag
    bad = err > bound
    assert not np.any(bad), (f"{what}: {int(bad.sum())} values outside tolerance; worst "
                             f"|d|={err[bad].max():.3e} at M={ref.mag[bad][np.argmax(err[bad])]:.3e}")
    return float(np.max(err / np.where(ref.mag > 0, ref.mag, 1.0))) if len(err) else 0.0


def row_ptr_sha256(rp) -> str:
    return hashlib.sha256(np.ascontiguousarray(rp, dtype="<i8").tobytes()).hexdigest()


def col_blocks_sha256_device(c_rp_host: np.ndarray, c_col_dev) -> str:
    """SHA-256 over the per-block SHA-256 of col_idx, blocks as defined by
    make_golden.col_blocks (computed from the row_ptr)."""
    digests = []
    for r0, r1 in make_golden.col_blocks(c_rp_host):
        a, b = int(c_rp_host[r0]), int(c_rp_host[r1])
        chunk = c_col_dev[a:b].cpu().numpy().astype("<i4", copy=False)
        digests.append(hashlib.sha256(chunk.tobytes()).digest())
    return hashlib.sha256(b"".join(digests)).hexdigest()
