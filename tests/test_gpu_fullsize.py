"""Full-size parity on the two R-MAT workloads, in the default launch
configuration the benchmark times.

The whole structure is compared bit for bit with the oracle through the
digests in tests/golden/oracle_summaries.txt (written from the oracle by
tests/golden/make_golden.py): SHA-256 of C.row_ptr and a block-wise SHA-256
of C.col_idx. Values are compared with the oracle itself on a sample of
rows: the heaviest rows plus random rows from every size class.
"""
import numpy as np
import pytest

import matgen
import oracle
from gpu_util import assert_matches, col_blocks_sha256_device, golden, row_ptr_sha256

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def sample_rows(prods: np.ndarray, seed: int, per_class: int = 40, top: int = 6) -> np.ndarray:
    rng = np.random.default_rng(seed)
    rows = list(np.argsort(prods)[::-1][:top])
    edges = [1, 65, 1025, 16385, 262145, 1 << 62]
    for lo, hi in zip(edges[:-1], edges[1:]):
        cand = np.nonzero((prods >= lo) & (prods < hi))[0]
        if len(cand):
            rows += list(rng.choice(cand, size=min(per_class, len(cand)), replace=False))
    rows += list(rng.choice(len(prods), size=20, replace=False))   # includes empty rows
    return np.array(sorted(set(int(r) for r in rows)), dtype=np.int64)


def run_full(name: str, seed: int):
    import torch
    from paper_2606_20855_amd import wingspan as ws

    g = golden(name)
    if not g or "col_blocks_sha256" not in g:
        pytest.skip(f"no oracle summary for {name}")
    A, B = matgen.config(name)
    print(f"{name}: m={A.nrows} nnz={A.nnz}", flush=True)
    dA = ws.DeviceCSR.from_host(A, "cuda:0")
    C = ws.spgemm(dA, dA)
    torch.cuda.synchronize()
    sym, num = ws.wingspan_last_stats(0), ws.wingspan_last_stats(1)
    print(f"{name}: symbolic {sym['rows']} numeric {num['rows']}", flush=True)
    rp = C.row_ptr.cpu().numpy()
    assert sym["total_products"] == g["products"]
    assert int(rp[-1]) == g["nnz_c"]
    assert row_ptr_sha256(rp) == g["row_ptr_sha256"]
    assert col_blocks_sha256_device(rp, C.col_idx) == g["col_blocks_sha256"]
    print(f"{name}: structure matches the oracle digests", flush=True)

    prods = oracle.row_products(A, A)
    rows = sample_rows(prods, seed)
    ref = oracle.spgemm(A, A, rows=rows)
    segs = [(int(rp[i]), int(rp[i + 1])) for i in rows]
    sub_rp = np.zeros(len(rows) + 1, dtype=np.int64)
    sub_rp[1:] = np.cumsum([b - a for a, b in segs])
    col = torch.cat([C.col_idx[a:b] for a, b in segs]).cpu().numpy()
    val = torch.cat([C.val[a:b] for a, b in segs]).cpu().numpy()
    got = ws.HostCSR(len(rows), A.ncols, sub_rp, col, val)
    worst = assert_matches(got, ref, A.val.dtype, what=f"{name} sampled rows")
    print(f"{name}: {len(rows)} sampled rows ({ref.nnz} entries) within tolerance, worst |d|/M = {worst:.2e}",
          flush=True)
    return num


def test_rmat18_full_size():
    num = run_full("rmat18", 1818)
    assert num["rows"]["dense"] > 0


def test_rmat20_full_size():
    run_full("rmat20", 2020)
