"""Write tests/golden/oracle_summaries.txt from the CPU oracle.

Calls only the oracle (oracle/) and the seeded generators (matgen/). For each
named workload it records the sizes, the total product count P, nnz(C), a
SHA-256 of C.row_ptr (int64, little endian) and a SHA-256 over blocks of
C.col_idx (int32, little endian). Column blocks are the row ranges obtained by
cutting C.row_ptr greedily at the first row boundary at or after every
multiple of BLOCK_ENTRIES entries; the digest is SHA-256 over the
concatenated per-block digests. The GPU tests recompute both digests from
their own output and compare.

Usage: python tests/golden/make_golden.py [config ...]   (default: all)
"""
from __future__ import annotations

import hashlib
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import matgen  # noqa: E402
import oracle  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_summaries.txt")
BLOCK_ENTRIES = 1 << 26
_A = _B = None


def col_blocks(row_ptr: np.ndarray, block_entries: int = BLOCK_ENTRIES):
    """Row ranges [r0, r1) cutting row_ptr at the first row boundary at or
    after each multiple of block_entries."""
    m = len(row_ptr) - 1
    blocks, r0 = [], 0
    while r0 < m:
        target = row_ptr[r0] + block_entries
        r1 = int(np.searchsorted(row_ptr, target, side="left"))
        r1 = max(r1, r0 + 1)
        r1 = min(r1, m)
        blocks.append((r0, r1))
        r0 = r1
    return blocks


def _count_chunk(rng):
    r0, r1 = rng
    res = oracle.spgemm(_A, _B, rows=np.arange(r0, r1, dtype=np.int64), with_mag=False)
    return r0, np.diff(res.row_ptr)


def _hash_block(rng):
    r0, r1 = rng
    res = oracle.spgemm(_A, _B, rows=np.arange(r0, r1, dtype=np.int64), with_mag=False)
    return r0, hashlib.sha256(np.ascontiguousarray(res.col_idx, dtype="<i4").tobytes()).digest()


def _chunks_by_products(prods: np.ndarray, target: int):
    cum = np.cumsum(prods)
    out, r0 = [], 0
    m = len(prods)
    while r0 < m:
        base = cum[r0 - 1] if r0 else 0
        r1 = int(np.searchsorted(cum, base + target, side="right"))
        r1 = min(max(r1, r0 + 1), m)
        out.append((r0, r1))
        r0 = r1
    return out


def summarize(name: str, workers: int) -> dict:
    global _A, _B
    t0 = time.time()
    _A, _B = matgen.config(name)
    prods = oracle.row_products(_A, _B)
    P = int(prods.sum())
    chunks = _chunks_by_products(prods, max(1 << 22, P // (workers * 64)))
    counts = np.zeros(_A.nrows, dtype=np.int64)
    with mp.get_context("fork").Pool(workers) as pool:
        for r0, c in pool.imap_unordered(_count_chunk, chunks):
            counts[r0:r0 + len(c)] = c
        rp = np.zeros(_A.nrows + 1, dtype=np.int64)
        np.cumsum(counts, out=rp[1:])
        blocks = col_blocks(rp)
        digests = {}
        for r0, d in pool.imap_unordered(_hash_block, blocks):
            digests[r0] = d
    col_digest = hashlib.sha256(b"".join(digests[b[0]] for b in blocks)).hexdigest()
    s = dict(
        name=name,
        nrows=_A.nrows, ncols_a=_A.ncols, ncols_b=_B.ncols,
        nnz_a=_A.nnz, nnz_b=_B.nnz,
        dtype=str(_A.val.dtype),
        products=P,
        max_row_products=int(prods.max()) if len(prods) else 0,
        nnz_c=int(rp[-1]),
        max_row_nnz_c=int(counts.max()) if len(counts) else 0,
        row_ptr_sha256=hashlib.sha256(rp.astype("<i8").tobytes()).hexdigest(),
        col_blocks=len(blocks),
        col_blocks_sha256=col_digest,
    )
    print(f"{name}: {s} ({time.time() - t0:.1f}s)", flush=True)
    return s


def read(path: str = OUT) -> dict:
    out, cur = {}, None
    if not os.path.exists(path):
        return out
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("[") and line.endswith("]"):
            cur = out.setdefault(line[1:-1], {})
            continue
        k, v = line.split(":", 1)
        v = v.strip()
        cur[k.strip()] = int(v) if v.lstrip("-").isdigit() else v
    return out


def write(all_s: dict, path: str = OUT):
    with open(path, "w") as f:
        f.write("# Written by tests/golden/make_golden.py from the CPU oracle (oracle/) and the\n")
        f.write("# seeded generators (matgen/). Do not edit by hand.\n")
        f.write(f"# block_entries: {BLOCK_ENTRIES}\n")
        for name in matgen.CONFIGS:
            if name not in all_s:
                continue
            f.write(f"\n[{name}]\n")
            for k, v in all_s[name].items():
                if k != "name":
                    f.write(f"{k}: {v}\n")


if __name__ == "__main__":
    names = sys.argv[1:] or list(matgen.CONFIGS)
    workers = int(os.environ.get("GOLDEN_WORKERS", min(8, os.cpu_count() or 1)))
    current = read()
    for nm in names:
        current[nm] = summarize(nm, workers)
        write(current)
