"""A seeded random sweep of inputs and options against the oracle.

Each case draws a matrix pair (Bernoulli, R-MAT or striped columns, square
or rectangular, narrow or wider than one 262,144-column region), a value type
and a set of options that route rows to particular tiers (register, LDS hash,
dense bitmap / rank kernel, global spill), set window widths or the structure
cache's budget. The two-phase product and, for every third case, the single
pass must equal the oracle's C: structure bit for bit, values within the
tolerance of the value type. The cases are fixed by their index, so a failure
names one case that can be run on its own."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
import oracle
from gpu_util import assert_matches

pytestmark = pytest.mark.gpu

NCASES = 120

OPTION_SETS = [
    {},
    dict(tiny_max=-1),
    dict(tiny_max=-1, max_lds_slots=64),
    dict(tiny_max=-1, max_lds_slots=64, cache_mib=-1),
    dict(tiny_max=-1, max_lds_slots=64, cache_mib=1),
    dict(max_lds_slots=256, dense_min_nnz=1),
    dict(window_cols=1024, tiny_max=-1, max_lds_slots=64),
    dict(window_cols=4096),
    dict(force_spill=1),
    dict(dense_min_nnz=-1),
    dict(tiny_max=-1, max_lds_slots=64, wide_offsets=1),
]


def _striped(m, n, seed, dtype):
    rng = np.random.default_rng(seed)
    rows = []
    for _ in range(m):
        s = int(rng.choice([1, 2, 3, 7, 40]))
        cnt = int(rng.integers(0, max(2, min(n // s, 600))))
        lo = int(rng.integers(0, max(1, n - cnt * s)))
        rows.append(np.arange(lo, min(n, lo + cnt * s), s))
    rp = np.zeros(m + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32) if m else np.zeros(0, np.int32)
    val = rng.uniform(-1, 1, len(ci)) if dtype == np.float64 else 1.0 - rng.random(len(ci))
    return matgen.CSR(m, n, rp, ci, val.astype(dtype))


def draw_case(i: int):
    rng = np.random.default_rng(1000 + i)
    dtype = np.float32 if rng.random() < 0.5 else np.float64
    dist = "open01" if dtype == np.float32 else "pm1"
    kind = ["bernoulli", "rmat", "striped", "wide"][i % 4]
    if kind == "bernoulli":
        m, k, n = (int(x) for x in rng.integers(1, 400, 3))
        A = matgen.random_sparse(m, k, float(rng.uniform(0.005, 0.3)), seed=2000 + i, dtype=dtype, dist=dist,
                                 empty_rows=float(rng.uniform(0, 0.3)))
        B = matgen.random_sparse(k, n, float(rng.uniform(0.005, 0.3)), seed=3000 + i, dtype=dtype, dist=dist)
    elif kind == "rmat":
        A = matgen.rmat(int(rng.integers(7, 11)), int(rng.integers(4, 17)), seed=4000 + i, dtype=dtype, dist=dist)
        B = A
    elif kind == "striped":
        k = int(rng.integers(20, 200))
        n = int(rng.integers(1000, 60000))
        B = _striped(k, n, 5000 + i, dtype)
        A = matgen.random_sparse(int(rng.integers(1, 120)), k, float(rng.uniform(0.02, 0.3)), seed=6000 + i,
                                 dtype=dtype, dist=dist)
    else:
        # columns past one rank region (262,144)
        n = int(rng.integers(262_145, 700_000))
        A = matgen.er(int(rng.integers(4, 40)), 600, int(rng.integers(20, 200)), seed=7000 + i, dtype=dtype, dist=dist)
        B = matgen.er(600, n, int(rng.integers(5, 60)), seed=8000 + i, dtype=dtype, dist=dist)
    opts = OPTION_SETS[int(rng.integers(0, len(OPTION_SETS)))]
    return kind, A, B, opts


@pytest.mark.parametrize("i", range(NCASES))
def test_random_case(i):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    kind, A, B, opts = draw_case(i)
    print(f"sweep case {i}: {kind} A {A.nrows}x{A.ncols} nnz={A.nnz} B {B.nrows}x{B.ncols} nnz={B.nnz} "
          f"dtype={A.val.dtype} options={opts}", flush=True)
    ref = oracle.spgemm(A, B)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    dB = dA if B is A else ws.DeviceCSR.from_host(B, "cuda:0")
    got = ws.spgemm(dA, dB, options=dict(opts) or None)
    torch.cuda.synchronize()
    assert_matches(got.to_host(), ref, A.val.dtype, what=f"case {i} two-phase")
    if i % 3 == 0:
        S = ws.spgemm_sharded(dA, dB, options=dict(opts) or None)
        got2 = ws.sharded_to_csr(S)
        torch.cuda.synchronize()
        assert_matches(got2.to_host(), ref, A.val.dtype, what=f"case {i} single pass")
