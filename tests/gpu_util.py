"""Helpers for the GPU parity tests: run the library through the C ABI and
compare its output with the CPU oracle."""
from __future__ import annotations

import hashlib
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

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


def gpu_row_products(A, B) -> np.ndarray:
    """Per-row product counts of C = A * B from the library's analysis pass
    (wingspan_spgemm_row_products through the C ABI), on cuda:0."""
    import torch
    from paper_2606_20855_amd import wingspan as ws

    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")
    out = ws.row_products(dA, dB)
    torch.cuda.synchronize()
    return out.cpu().numpy()


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


def product_blocks(prods: np.ndarray, r0: int, r1: int, target: int):
    """Row ranges covering [r0, r1), each holding about `target` products (at
    least one row)."""
    cum = np.cumsum(prods[r0:r1], dtype=np.int64)
    out, a = [], 0
    n = r1 - r0
    while a < n:
        base = cum[a - 1] if a else 0
        b = int(np.searchsorted(cum, base + target, side="right"))
        b = min(max(b, a + 1), n)
        out.append((r0 + a, r0 + b))
        a = b
    return out


def compare_rows(A, B, rp, r0, r1, col, val, prods):
    """Rows [r0, r1) of C (row pointer rp, host int64; col and val the host
    copies of entries [rp[r0], rp[r1])) against the oracle: lengths and
    columns bit for bit, values within tol * M (exactly zero where M = 0).
    Returns (entries, worst |d|/M)."""
    rows = np.arange(r0, r1, dtype=np.int64)
    bound = int(np.minimum(prods[r0:r1], B.ncols).sum())
    ref = oracle_spgemm(A, B, rows, bound)
    what = f"rows [{r0}, {r1})"
    lens = np.diff(rp[r0:r1 + 1])
    if not np.array_equal(lens, np.diff(ref.row_ptr)):
        bad = int(np.nonzero(lens != np.diff(ref.row_ptr))[0][0]) + r0
        raise AssertionError(f"{what}: row {bad} has {int(rp[bad + 1] - rp[bad])} entries, the oracle "
                             f"{int(ref.row_ptr[bad - r0 + 1] - ref.row_ptr[bad - r0])}")
    if not np.array_equal(col, ref.col_idx):
        p = int(np.nonzero(col != ref.col_idx)[0][0])
        raise AssertionError(f"{what}: col_idx differs first at entry {int(rp[r0]) + p}")
    tol = TOL[np.dtype(A.val.dtype)]
    err = np.abs(val.astype(np.float64) - ref.val.astype(np.float64))
    bound_v = tol * ref.mag
    bad = err > bound_v
    if np.any(bad):
        k = int(np.argmax(bad))
        raise AssertionError(f"{what}: {int(bad.sum())} values outside tolerance; first at entry "
                             f"{int(rp[r0]) + k}: gpu {val[k]!r} oracle {ref.val[k]!r} M {ref.mag[k]:.3e}")
    worst = float(np.max(err / np.where(ref.mag > 0, ref.mag, 1.0))) if len(err) else 0.0
    return len(err), worst


def oracle_spgemm(A, B, rows, capacity):
    import oracle
    return oracle.spgemm(A, B, rows=rows, capacity=capacity)


def check_rows_blockwise(A, B, rp, fetch, ranges=None, workers=None, block_products=1 << 25, log=None):
    """Every row in `ranges` (list of [r0, r1), default all rows) of C against
    the oracle, block by block on `workers` host threads (the oracle is C
    called through ctypes, which releases the interpreter lock). fetch(a, b)
    returns the host (col, val) of C's entries [a, b). Returns a summary dict;
    raises AssertionError at the first mismatch."""
    import oracle
    t0 = time.time()
    workers = workers or min(16, os.cpu_count() or 1)
    ranges = ranges if ranges is not None else [(0, A.nrows)]
    prods = oracle.row_products(A, B)
    blocks = [blk for r0, r1 in ranges if r1 > r0 for blk in product_blocks(prods, r0, r1, block_products)]

    def work(blk):
        r0, r1 = blk
        col, val = fetch(int(rp[r0]), int(rp[r1]))
        return compare_rows(A, B, rp, r0, r1, col, val, prods)

    entries, worst, done, last = 0, 0.0, 0, t0
    with ThreadPoolExecutor(workers) as ex:
        for n, w in ex.map(work, blocks):
            entries += n
            worst = max(worst, w)
            done += 1
            if log and (time.time() - last > 10 or done == len(blocks)):
                last = time.time()
                log(f"  {done}/{len(blocks)} blocks, {entries} entries within tolerance "
                    f"({time.time() - t0:.0f} s)")
    rows = sum(r1 - r0 for r0, r1 in ranges)
    return dict(rows=rows, entries=entries, worst=worst, blocks=len(blocks), seconds=time.time() - t0,
                products=int(sum(prods[r0:r1].sum() for r0, r1 in ranges)))
