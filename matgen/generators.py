"""Seeded generators for the SpGEMM workloads.

The paper evaluates SpGEMM on randomly generated matrices with a fixed
number of nonzeros per row (Section 5.1, scaling figure) and on the
SuiteSparse/SNAP matrices of Zhang et al. Those matrices are not available
here, so synthetic stand-ins are generated with the same structure:

* Erdos-Renyi rows with exactly ``r`` distinct uniformly random columns
  (the paper's own fixed-nnz-per-row random matrices),
* the 2D 5-point Laplacian (mesh / PDE matrices),
* R-MAT power-law graphs (heavy-tailed SNAP-like graphs),
* a rectangular Erdos-Renyi product (non-square shapes).

Readings of details the workload descriptions leave open:

* R-MAT: one quadrant draw per bit, most significant bit first; quadrant
  ``a`` -> (row bit 0, col bit 0), ``b`` -> (0, 1), ``c`` -> (1, 0),
  ``d`` -> (1, 1). No noise, no vertex permutation, directed edges. Exactly
  ``edge_factor * 2**scale`` edges are drawn, duplicates are merged into one
  entry and self-loops are kept. One value is drawn per surviving entry in
  CSR order (duplicates are not summed).
* fp64 values "uniform in [-1, 1]" are ``2U - 1`` with ``U`` a 53-bit uniform
  in [0, 1). fp32 values "uniform in (0, 1]" are ``1 - k * 2**-24`` with ``k``
  uniform in [0, 2**24): exactly representable and never zero.
* Erdos-Renyi rows hold exactly ``r`` distinct columns sampled without
  replacement, sorted.
* The Laplacian has Dirichlet boundaries (missing neighbours are dropped),
  natural ordering ``p = x + g*y``, 4 on the diagonal and -1 off it.

All randomness comes from ``numpy.random.Generator(PCG64(seed))``.
"""
from __future__ import annotations

import numpy as np

from .csr import CSR

_U24 = float(2.0 ** -24)


def _rng(seed) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _values(rng: np.random.Generator, n: int, dist: str, dtype) -> np.ndarray:
    if dist == "pm1":
        v = 2.0 * rng.random(n) - 1.0
    elif dist == "open01":
        k = rng.integers(0, 1 << 24, size=n, dtype=np.int64)
        v = 1.0 - k.astype(np.float64) * _U24
    elif dist == "ones":
        v = np.ones(n)
    elif dist == "int":
        v = rng.integers(1, 4, size=n).astype(np.float64)
    else:
        raise ValueError(f"unknown value distribution {dist!r}")
    return v.astype(dtype)


def _csr_from_sorted_keys(keys: np.ndarray, nrows: int, ncols: int) -> tuple:
    """keys = row*ncols + col, strictly increasing."""
    rows = keys // ncols
    cols = (keys - rows * ncols).astype(np.int32)
    counts = np.bincount(rows, minlength=nrows)
    rp = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(counts, out=rp[1:])
    return rp.astype(np.int32), cols


def er(m: int, n: int, r: int, seed, dtype=np.float64, dist: str = "pm1") -> CSR:
    """m x n, every row holds exactly r distinct uniformly random columns."""
    if r > n:
        raise ValueError("r > n")
    rng = _rng(seed)
    if r * r > n:
        # a row of r independent draws would almost surely repeat a column:
        # draw each row without replacement instead
        cols = np.stack([np.sort(rng.choice(n, size=r, replace=False)) for _ in range(m)]).astype(np.int64)
        cols = cols.reshape(m, r)
        rp = (np.arange(m + 1, dtype=np.int64) * r).astype(np.int32)
        val = _values(rng, m * r, dist, dtype)
        return CSR(m, n, rp, cols.reshape(-1).astype(np.int32), val)
    cols = np.sort(rng.integers(0, n, size=(m, r), dtype=np.int64), axis=1)
    # redraw rows that picked a column twice until every row is distinct
    while True:
        bad = np.nonzero(np.any(np.diff(cols, axis=1) == 0, axis=1))[0] if r > 1 else np.zeros(0, np.int64)
        if len(bad) == 0:
            break
        cols[bad] = np.sort(rng.integers(0, n, size=(len(bad), r), dtype=np.int64), axis=1)
    rp = (np.arange(m + 1, dtype=np.int64) * r).astype(np.int32)
    val = _values(rng, m * r, dist, dtype)
    return CSR(m, n, rp, cols.reshape(-1).astype(np.int32), val)


def laplacian2d(g: int, dtype=np.float64) -> CSR:
    """5-point stencil on a g x g grid, Dirichlet boundary, p = x + g*y."""
    n = g * g
    p = np.arange(n, dtype=np.int64)
    x, y = p % g, p // g
    # neighbours in increasing column order: up (p-g), left (p-1), self, right (p+1), down (p+g)
    cand = np.stack([p - g, p - 1, p, p + 1, p + g], axis=1)
    ok = np.stack([y > 0, x > 0, np.ones(n, bool), x < g - 1, y < g - 1], axis=1)
    vals = np.where(cand == p[:, None], 4.0, -1.0)
    counts = ok.sum(axis=1)
    rp = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(counts, out=rp[1:])
    return CSR(n, n, rp.astype(np.int32), cand[ok].astype(np.int32), vals[ok].astype(dtype))


def rmat(scale: int, edge_factor: int = 16, abcd=(0.57, 0.19, 0.19, 0.05), seed=0,
         dtype=np.float32, dist: str = "open01") -> CSR:
    """Directed R-MAT graph with 2**scale vertices and edge_factor*2**scale
    drawn edges, duplicates merged, self-loops kept."""
    a, b, c, d = abcd
    if abs(a + b + c + d - 1.0) > 1e-9:
        raise ValueError("quadrant probabilities must sum to 1")
    nv = 1 << scale
    ne = edge_factor * nv
    rng = _rng(seed)
    rows = np.zeros(ne, dtype=np.int64)
    cols = np.zeros(ne, dtype=np.int64)
    t_ab, t_abc = a + b, a + b + c
    for lvl in range(scale):
        bit = np.int64(1) << np.int64(scale - 1 - lvl)
        u = rng.random(ne)
        rbit = u >= t_ab                     # quadrants c, d
        cbit = ((u >= a) & (u < t_ab)) | (u >= t_abc)   # quadrants b, d
        rows += rbit * bit
        cols += cbit * bit
    keys = np.unique(rows * nv + cols)
    del rows, cols
    rp, ci = _csr_from_sorted_keys(keys, nv, nv)
    val = _values(rng, len(ci), dist, dtype)
    return CSR(nv, nv, rp, ci, val)


def er_rect(m: int, k: int, n: int, r: int, seed, dtype=np.float64, dist: str = "pm1"):
    """A (m x k) and B (k x n), both with exactly r distinct columns per row."""
    sa, sb = np.random.SeedSequence(seed).spawn(2)
    return er(m, k, r, sa, dtype, dist), er(k, n, r, sb, dtype, dist)


def arrowhead(n: int, dtype=np.float64) -> CSR:
    """Ones on the first row, the first column and the diagonal."""
    rows, cols = [], []
    rows.append(np.zeros(n, np.int64)); cols.append(np.arange(n, dtype=np.int64))
    rows.append(np.arange(1, n, dtype=np.int64)); cols.append(np.zeros(n - 1, np.int64))
    rows.append(np.arange(1, n, dtype=np.int64)); cols.append(np.arange(1, n, dtype=np.int64))
    keys = np.unique(np.concatenate(rows) * n + np.concatenate(cols))
    rp, ci = _csr_from_sorted_keys(keys, n, n)
    return CSR(n, n, rp, ci, np.ones(len(ci), dtype=dtype))


def shuffled_copy(M: CSR, seed) -> CSR:
    """M with its rows and columns relabelled by two seeded random
    permutations (B[p(i), q(j)] = M[i, j]): the same values and degree
    distribution on a different pattern."""
    rng = _rng(seed)
    p = rng.permutation(M.nrows).astype(np.int64)
    q = rng.permutation(M.ncols).astype(np.int64)
    rows = np.repeat(np.arange(M.nrows, dtype=np.int64), np.diff(M.row_ptr))
    keys = p[rows] * max(M.ncols, 1) + q[M.col_idx.astype(np.int64)]
    order = np.argsort(keys)   # the keys are distinct, so any sort gives this order
    rp, ci = _csr_from_sorted_keys(keys[order], M.nrows, M.ncols)
    return CSR(M.nrows, M.ncols, rp, ci, M.val[order].copy())


def transpose(M: CSR) -> CSR:
    """The CSR arrays of M's transpose (equivalently, M in compressed
    columns): the same entries, grouped by column, rows ascending."""
    rows = np.repeat(np.arange(M.nrows, dtype=np.int64), np.diff(M.row_ptr))
    keys = M.col_idx.astype(np.int64) * max(M.nrows, 1) + rows
    order = np.argsort(keys)   # distinct keys
    rp, ci = _csr_from_sorted_keys(keys[order], M.ncols, M.nrows)
    return CSR(M.ncols, M.nrows, rp, ci, M.val[order].copy())


def sparse_vector(n: int, density: float, seed, dtype=np.float64, dist: str = "pm1"):
    """A seeded sparse vector of length n: round(density * n) distinct
    indices drawn uniformly (returned sorted, int32) and their values."""
    rng = _rng(seed)
    k = int(round(density * n))
    idx = np.sort(rng.choice(n, size=k, replace=False)).astype(np.int32) if k > 0 else np.zeros(0, np.int32)
    return idx, _values(rng, k, dist, dtype)


def identity(n: int, dtype=np.float64) -> CSR:
    return CSR(n, n, np.arange(n + 1, dtype=np.int32), np.arange(n, dtype=np.int32),
               np.ones(n, dtype=dtype))


def permutation(n: int, seed, dtype=np.float64) -> CSR:
    """Row i holds a single one at column perm[i]."""
    perm = _rng(seed).permutation(n)
    return CSR(n, n, np.arange(n + 1, dtype=np.int32), perm.astype(np.int32),
               np.ones(n, dtype=dtype))


def diagonal(d: np.ndarray) -> CSR:
    n = len(d)
    return CSR(n, n, np.arange(n + 1, dtype=np.int32), np.arange(n, dtype=np.int32), d.copy())


def random_sparse(m: int, n: int, density: float, seed, dtype=np.float64,
                  dist: str = "pm1", empty_rows: float = 0.0) -> CSR:
    """Bernoulli(density) pattern, optionally with a fraction of rows forced empty."""
    rng = _rng(seed)
    mask = rng.random((m, n)) < density
    if empty_rows > 0 and m > 0:
        mask[rng.random(m) < empty_rows] = False
    r, c = np.nonzero(mask)
    keys = r.astype(np.int64) * n + c
    rp, ci = _csr_from_sorted_keys(keys, m, n) if n > 0 else (np.zeros(m + 1, np.int32), np.zeros(0, np.int32))
    val = _values(rng, len(ci), dist, dtype)
    return CSR(m, n, rp, ci, val)


# ---------------------------------------------------------------------------
# The five named workloads. Each returns (A, B); C = A @ B.
# ---------------------------------------------------------------------------

def _cfg_er1000(seed=1):
    A = er(1000, 1000, 10, seed, np.float64, "pm1")
    return A, A


def _cfg_laplace512(seed=None):
    A = laplacian2d(512, np.float64)
    return A, A


def _cfg_rmat18(seed=18):
    A = rmat(18, 16, (0.57, 0.19, 0.19, 0.05), seed, np.float32, "open01")
    return A, A


def _cfg_er_rect(seed=4):
    return er_rect(1_000_000, 500_000, 1_000_000, 8, seed, np.float64, "pm1")


def _cfg_rmat20(seed=20):
    A = rmat(20, 16, (0.57, 0.19, 0.19, 0.05), seed, np.float64, "pm1")
    return A, A


def _cfg_rmat22(seed=22):
    A = rmat(22, 16, (0.57, 0.19, 0.19, 0.05), seed, np.float64, "pm1")
    return A, A


CONFIGS = {
    "er1000": dict(make=_cfg_er1000, seed=1, dtype="f64",
                   desc="C=A*A, Erdos-Renyi 1000x1000, 10 distinct nnz/row, fp64 U[-1,1]"),
    "laplace512": dict(make=_cfg_laplace512, seed=None, dtype="f64",
                       desc="C=A*A, 2D 5-point Laplacian on 512x512 grid, fp64"),
    "rmat18": dict(make=_cfg_rmat18, seed=18, dtype="f32",
                   desc="C=A*A, R-MAT scale 18, edge factor 16, (.57,.19,.19,.05), fp32 (0,1]"),
    "er_rect": dict(make=_cfg_er_rect, seed=4, dtype="f64",
                    desc="C=A*B, A 1e6x5e5 and B 5e5x1e6 Erdos-Renyi, 8 distinct nnz/row, fp64"),
    "rmat20": dict(make=_cfg_rmat20, seed=20, dtype="f64",
                   desc="C=A*A, R-MAT scale 20, edge factor 16, (.57,.19,.19,.05), fp64 U[-1,1]"),
}

# Single matrices that no product is formed from: the larger input of the
# elementwise and SpMSpV measurements.
MATRICES = {
    "rmat22": dict(make=_cfg_rmat22, seed=22, dtype="f64",
                   desc="R-MAT scale 22, edge factor 16, (.57,.19,.19,.05), fp64 U[-1,1]"),
}


def matrix(name: str):
    """A named workload's A: one of CONFIGS (its A) or of MATRICES."""
    if name in CONFIGS:
        return config(name)[0]
    cfg = MATRICES[name]
    return cfg["make"](cfg["seed"])[0]


def config(name: str):
    """Build the (A, B) pair of a named workload."""
    cfg = CONFIGS[name]
    if cfg["seed"] is None:
        return cfg["make"]()
    return cfg["make"](cfg["seed"])
