"""Dense-tier structure passes over B rows of every column density.

The passes that mark a row's columns in an LDS bitmap merge the bits of
neighbouring columns that share a 32-bit word before their atomics (pairs of
lanes, and runs inside a lane that holds four consecutive columns). B rows
with columns at strides 1, 2, 3, 5, 8 and 33, and random ones, make lanes
share words always, often, rarely or never. The column sets are formed three
ways: by the symbolic phase (kept for the numeric phase), by the numeric
phase's own structure pass (no cache), and by the single pass; each result
must equal the oracle's."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
import oracle
from gpu_util import assert_matches

pytestmark = pytest.mark.gpu

# rows above 42 output entries skip the LDS hash tiers
DENSE = dict(tiny_max=-1, max_lds_slots=64)
STRIDES = (1, 2, 3, 5, 8, 33)


def _values(rng, n, dtype):
    if dtype == np.float32:
        return (1.0 - rng.random(n)).astype(dtype)   # (0, 1]
    return rng.uniform(-1.0, 1.0, n).astype(dtype)


def striped_b(nrows: int, ncols: int, seed: int, dtype) -> matgen.CSR:
    """Row k: a run of columns at one of STRIDES from a random start (every
    seventh row: random distinct columns instead)."""
    rng = np.random.default_rng(seed)
    rows = []
    for k in range(nrows):
        if k % 7 == 6:
            rows.append(np.sort(rng.choice(ncols, 1500, replace=False)))
            continue
        s = STRIDES[k % len(STRIDES)]
        n = int(rng.integers(300, 3000))
        lo = int(rng.integers(0, max(1, ncols - n * s)))
        rows.append(np.arange(lo, min(ncols, lo + n * s), s))
    rp = np.zeros(nrows + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    return matgen.CSR(nrows, ncols, rp, ci, _values(rng, len(ci), dtype))


def picking_a(nrows: int, nb: int, per_row: int, seed: int, dtype) -> matgen.CSR:
    """Each row takes per_row distinct rows of B."""
    rng = np.random.default_rng(seed)
    cols = [np.sort(rng.choice(nb, per_row, replace=False)) for _ in range(nrows)]
    rp = np.arange(nrows + 1, dtype=np.int32) * per_row
    ci = np.concatenate(cols).astype(np.int32)
    return matgen.CSR(nrows, nb, rp, ci, _values(rng, len(ci), dtype))


def _inputs(dtype, seed):
    B = striped_b(60, 40_000, seed, dtype)
    A = picking_a(40, B.nrows, 10, seed + 1, dtype)
    return A, B


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("mode", ["cached", "uncached", "single_pass"])
def test_every_column_density(dtype, mode):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    A, B = _inputs(dtype, seed=71 if dtype == np.float32 else 73)
    print(f"bitmap density: mode={mode} dtype={np.dtype(dtype).name} nnz(A)={A.nnz} nnz(B)={B.nnz}", flush=True)
    ref = oracle.spgemm(A, B)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = ws.DeviceCSR.from_host(B, "cuda:0")
    if mode == "single_pass":
        S = ws.spgemm_sharded(dA, dB, options=dict(DENSE))
        st = ws.wingspan_last_stats(2)
        got = ws.sharded_to_csr(S)
    else:
        opts = dict(DENSE, cache_mib=-1) if mode == "uncached" else dict(DENSE)
        got = ws.spgemm(dA, dB, options=opts)
        st = ws.wingspan_last_stats(1)
        assert (st["structure_cache_rows"] == 0) == (mode == "uncached")
    torch.cuda.synchronize()
    assert st["rows"]["dense"] == A.nrows
    assert_matches(got.to_host(), ref, dtype, what=f"{mode} {np.dtype(dtype).name}")
