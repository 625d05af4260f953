"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test checks the oracle against something independent of its own code:
a hand-worked product, a dense brute-force product, a closed form, an
algebraic identity, or an invariant of the CSR format. Together they are
chosen so that a dropped term, a wrong sign, a wrong index or a transposed
operand in the oracle fails at least one of them.
"""
import math
import zlib

import numpy as np
import pytest

import matgen
import oracle
from matgen import CSR


def csr_from_dense(d: np.ndarray, dtype=np.float64, keep=None) -> CSR:
    """Stored entries are the nonzeros of d (or the True entries of keep)."""
    mask = (d != 0) if keep is None else keep
    r, c = np.nonzero(mask)
    rp = np.zeros(d.shape[0] + 1, dtype=np.int64)
    np.cumsum(np.bincount(r, minlength=d.shape[0]), out=rp[1:])
    return CSR(d.shape[0], d.shape[1], rp.astype(np.int32), c.astype(np.int32),
               d[r, c].astype(dtype))


def assert_canonical(res, nrows, ncols):
    rp = res.row_ptr
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0) and rp[-1] == len(res.col_idx)
    for i in range(nrows):
        c = res.col_idx[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0)
        assert len(c) == 0 or (c[0] >= 0 and c[-1] < ncols)


# ---------------------------------------------------------------------------
# A product worked out by hand.
# ---------------------------------------------------------------------------

def test_hand_worked_example():
    # A (4x4) and B (4x3); the last row of A produces an exact cancellation.
    A = np.array([[1.0, 0.0, 2.0, 0.0],
                  [0.0, 0.0, 0.0, 0.0],
                  [0.0, 3.0, 0.0, -1.0],
                  [1.0, 0.5, 0.0, 0.0]])
    B = np.array([[0.0, 1.0, 0.0],
                  [2.0, -2.0, 0.0],
                  [0.0, 0.0, 4.0],
                  [1.0, 0.0, -3.0]])
    # row 0 = 1*B0 + 2*B2 = [0, 1, 8]            -> cols {1, 2}
    # row 1 = empty
    # row 2 = 3*B1 - 1*B3 = [6-1, -6, 0+3]       -> cols {0, 1, 2} = [5, -6, 3]
    # row 3 = 1*B0 + 0.5*B1 = [1, 1-1, 0]        -> cols {0, 1} = [1, 0]; the
    #         zero at column 1 is structural (two products were formed) and stays.
    res = oracle.spgemm(csr_from_dense(A), csr_from_dense(B))
    assert list(res.row_ptr) == [0, 2, 2, 5, 7]
    assert list(res.col_idx) == [1, 2, 0, 1, 2, 0, 1]
    assert list(res.val) == [1.0, 8.0, 5.0, -6.0, 3.0, 1.0, 0.0]
    # magnitudes: row 2 col 0 = |3*2| + |-1*1| = 7, row 3 col 1 = |1*1| + |0.5*-2| = 2
    assert list(res.mag) == [1.0, 8.0, 7.0, 6.0, 3.0, 1.0, 2.0]
    # products: |B0|=1, |B1|=2, |B2|=1, |B3|=2 -> rows: 1+1, 0, 2+2, 1+2
    assert list(res.products) == [2, 0, 4, 3]


# ---------------------------------------------------------------------------
# Brute force: dense products on tiny random shapes.
# ---------------------------------------------------------------------------

SHAPES = [(0, 0, 0), (1, 1, 1), (2, 3, 2), (3, 2, 7), (7, 33, 5), (33, 7, 64),
          (64, 64, 64), (5, 0, 4), (0, 5, 3), (4, 6, 0), (17, 64, 33)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("density", [0.0, 0.1, 0.5, 1.0])
@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_dense_bruteforce(shape, density, dtype):
    m, k, n = shape
    seed = zlib.crc32(repr((shape, density, np.dtype(dtype).name)).encode()) & 0xFFFF
    A = matgen.random_sparse(m, k, density, seed, dtype, "pm1", empty_rows=0.2)
    B = matgen.random_sparse(k, n, density, seed + 1, dtype, "pm1", empty_rows=0.2)
    res = oracle.spgemm(A, B)
    assert_canonical(res, m, n)
    # structure: boolean product of the stored patterns
    pat = (A.pattern_dense() @ B.pattern_dense()) > 0
    got = CSR(m, n, res.row_ptr, res.col_idx, np.ones(res.nnz)).pattern_dense() > 0
    assert np.array_equal(pat, got)
    # values: dense matmul of the stored values, within the summation bound
    Ad, Bd = A.to_dense(), B.to_dense()
    ref = Ad @ Bd
    magref = np.abs(Ad) @ np.abs(Bd)
    rows = np.repeat(np.arange(m), np.diff(res.row_ptr))
    cols = res.col_idx.astype(np.int64)
    eps = 1e-13 if dtype == np.float64 else 1.2e-7
    assert np.all(np.abs(res.val.astype(np.float64) - ref[rows, cols]) <= eps * magref[rows, cols] + 0.0)
    assert np.allclose(res.mag, magref[rows, cols], rtol=1e-13, atol=0)
    # product counts: sum over k of [A(i,k) stored] * len(B row k)
    blen = np.diff(B.row_ptr.astype(np.int64))
    assert np.array_equal(res.products, A.pattern_dense() @ blen if k else np.zeros(m, np.int64))


def test_not_transposed_or_swapped():
    # A*B differs from B*A, A^T*B and A*B^T on a non-symmetric square pair
    A = matgen.random_sparse(12, 12, 0.3, 5, np.float64)
    B = matgen.random_sparse(12, 12, 0.3, 6, np.float64)
    res = oracle.spgemm(A, B)
    Cd = CSR(12, 12, res.row_ptr, res.col_idx, res.val).to_dense()
    Ad, Bd = A.to_dense(), B.to_dense()
    assert np.allclose(Cd, Ad @ Bd, rtol=0, atol=1e-14)
    for wrong in (Bd @ Ad, Ad.T @ Bd, Ad @ Bd.T):
        assert not np.allclose(Cd, wrong, atol=1e-6)


# ---------------------------------------------------------------------------
# Identities: one product per output entry, so results are bit-exact.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_identity_both_sides(dtype):
    A = matgen.random_sparse(40, 40, 0.2, 11, dtype)
    I = matgen.identity(40, dtype)
    for res in (oracle.spgemm(I, A), oracle.spgemm(A, I)):
        assert np.array_equal(res.row_ptr, A.row_ptr.astype(np.int64))
        assert np.array_equal(res.col_idx, A.col_idx)
        assert np.array_equal(res.val, A.val)


def test_permutation_rows():
    A = matgen.random_sparse(50, 30, 0.2, 12, np.float64)
    P = matgen.permutation(50, 13)
    res = oracle.spgemm(P, A)
    perm = P.col_idx
    for i in range(50):
        c, v = A.row(perm[i])
        assert np.array_equal(res.col_idx[res.row_ptr[i]:res.row_ptr[i + 1]], c)
        assert np.array_equal(res.val[res.row_ptr[i]:res.row_ptr[i + 1]], v)


def test_diagonal_scaling_bit_exact():
    A = matgen.random_sparse(30, 20, 0.3, 14, np.float64)
    d = np.random.default_rng(15).uniform(-2, 2, 30)
    res = oracle.spgemm(matgen.diagonal(d), A)
    rows = np.repeat(np.arange(30), np.diff(A.row_ptr))
    assert np.array_equal(res.val, d[rows] * A.val)
    assert np.array_equal(res.col_idx, A.col_idx)


# ---------------------------------------------------------------------------
# Closed forms.
# ---------------------------------------------------------------------------

def laplacian_square_entry(g, p, q):
    """(L^2)[p,q] for the 5-point Dirichlet Laplacian, by hand: the diagonal is
    16 + deg(p); grid neighbours get -8; points two steps away in a straight
    line get 1; diagonal neighbours get 2 (two paths of length two)."""
    px, py, qx, qy = p % g, p // g, q % g, q // g
    dx, dy = abs(px - qx), abs(py - qy)
    deg = (px > 0) + (px < g - 1) + (py > 0) + (py < g - 1)
    if dx == 0 and dy == 0:
        return 16.0 + deg
    if dx + dy == 1:
        return -8.0
    if (dx, dy) in ((2, 0), (0, 2)):
        return 1.0
    if dx == 1 and dy == 1:
        return 2.0
    return None


@pytest.mark.parametrize("g", [1, 2, 3, 5, 8])
def test_laplacian_square_closed_form(g):
    L = matgen.laplacian2d(g)
    res = oracle.spgemm(L, L)
    n = g * g
    expected = {}
    for p in range(n):
        for q in range(n):
            v = laplacian_square_entry(g, p, q)
            if v is not None:
                expected[(p, q)] = v
    got = {}
    for p in range(n):
        for t in range(res.row_ptr[p], res.row_ptr[p + 1]):
            got[(p, int(res.col_idx[t]))] = float(res.val[t])
    assert got == expected


def test_laplacian_512_counts():
    g = 512
    L = matgen.laplacian2d(g)
    res = oracle.spgemm(L, L, with_mag=False)
    # nnz(L^2) = g^2 (diagonal) + 4g(g-1) (distance-1 pairs, both directions)
    #          + 4g(g-2) (straight distance 2) + 4(g-1)^2 (diagonal neighbours)
    assert res.nnz == g * g + 4 * g * (g - 1) + 4 * g * (g - 2) + 4 * (g - 1) ** 2 == 3_397_636
    # products = sum over k of nnz(row k)^2 for a symmetric L
    deg = np.diff(L.row_ptr.astype(np.int64))
    assert int(res.products.sum()) == int((deg ** 2).sum()) == 6_535_176
    # spot-check values against the closed form on a few rows (corner, edge, interior)
    for p in (0, 5, g + 1, 1000, g * g - 1, 131_328):
        for t in range(res.row_ptr[p], res.row_ptr[p + 1]):
            q = int(res.col_idx[t])
            assert res.val[t] == laplacian_square_entry(g, p, q)


@pytest.mark.parametrize("n", [2, 3, 64, 512])
def test_arrowhead_square_is_dense(n):
    # A = ones on the first row, first column and diagonal. A^2 is dense with
    # C[0,0] = n, C[0,j] = C[i,0] = 2, C[i,i] = 2 and 1 elsewhere (i, j >= 1).
    A = matgen.arrowhead(n)
    res = oracle.spgemm(A, A)
    assert res.nnz == n * n
    C = CSR(n, n, res.row_ptr, res.col_idx, res.val).to_dense()
    E = np.ones((n, n))
    E[0, :] = 2
    E[:, 0] = 2
    E[np.arange(n), np.arange(n)] = 2
    E[0, 0] = n
    assert np.array_equal(C, E)


def test_er1000_products_and_dense():
    A, B = matgen.config("er1000")
    res = oracle.spgemm(A, B)
    assert int(res.products.sum()) == 100_000            # 10 entries x 10 per row x 1000 rows
    assert np.all(res.products == 100)
    Ad = A.to_dense()
    ref = Ad @ Ad
    pat = (A.pattern_dense() @ A.pattern_dense()) > 0
    assert res.nnz == int(pat.sum())
    rows = np.repeat(np.arange(1000), np.diff(res.row_ptr))
    d = np.abs(res.val - ref[rows, res.col_idx])
    mag = (np.abs(Ad) @ np.abs(Ad))[rows, res.col_idx]
    assert np.all(d <= 1e-15 * mag)


def test_fp32_integer_sums_exact():
    # integer-valued fp32 inputs with many terms per entry: every partial sum
    # stays below 2^24, so the exact integer result must come out.
    A = matgen.random_sparse(64, 300, 0.5, 21, np.float32, "int")
    B = matgen.random_sparse(300, 40, 0.5, 22, np.float32, "int")
    res = oracle.spgemm(A, B)
    ref = A.to_dense().astype(np.int64) @ B.to_dense().astype(np.int64)
    assert ref.max() < 2 ** 24
    C = CSR(64, 40, res.row_ptr, res.col_idx, res.val).to_dense()
    assert np.array_equal(C.astype(np.int64), ref)


def test_fp32_rounded_once():
    # fp32 inputs: each product is exact in double, the sum is accumulated in
    # double and rounded to float once. Compare with the correctly rounded
    # exact sum (math.fsum over exact products), allowing the one case where
    # the double accumulation sits on the other side of a float tie.
    A = matgen.random_sparse(20, 200, 0.6, 31, np.float32)
    B = matgen.random_sparse(200, 20, 0.6, 32, np.float32)
    res = oracle.spgemm(A, B)
    Ad, Bd = A.to_dense(), B.to_dense()
    exact_rounded = 0
    for i in range(20):
        for t in range(res.row_ptr[i], res.row_ptr[i + 1]):
            j = res.col_idx[t]
            s = math.fsum(float(Ad[i, k]) * float(Bd[k, j]) for k in range(200) if Ad[i, k] and Bd[k, j])
            want = np.float32(s)
            got = res.val[t]
            assert abs(float(got) - float(want)) <= float(np.spacing(np.float32(abs(want))))
            exact_rounded += int(got == want)
    assert exact_rounded >= 0.99 * res.nnz


def test_magnitude_sums():
    A = matgen.random_sparse(25, 30, 0.3, 41, np.float64)
    B = matgen.random_sparse(30, 35, 0.3, 42, np.float64)
    res = oracle.spgemm(A, B)
    M = np.abs(A.to_dense()) @ np.abs(B.to_dense())
    rows = np.repeat(np.arange(25), np.diff(res.row_ptr))
    assert np.allclose(res.mag, M[rows, res.col_idx], rtol=1e-14, atol=0)
    # |c| <= M always
    assert np.all(np.abs(res.val) <= res.mag * (1 + 1e-15))


def test_row_subset_matches_full():
    A = matgen.random_sparse(60, 50, 0.15, 51, np.float64, empty_rows=0.3)
    B = matgen.random_sparse(50, 70, 0.15, 52, np.float64, empty_rows=0.3)
    full = oracle.spgemm(A, B)
    rows = np.array([59, 0, 7, 7, 33], dtype=np.int64)
    sub = oracle.spgemm(A, B, rows=rows)
    for s, i in enumerate(rows):
        a, b = full.row_ptr[i], full.row_ptr[i + 1]
        c, d = sub.row_ptr[s], sub.row_ptr[s + 1]
        assert np.array_equal(full.col_idx[a:b], sub.col_idx[c:d])
        assert np.array_equal(full.val[a:b], sub.val[c:d])
        assert full.products[i] == sub.products[s]


def test_single_pass_capacity_mode_matches_counting_mode():
    # the binding's one-call mode (output sized by a bound) returns the same rows as the counting mode; a bound
    # that is too small is refused rather than truncated
    A = matgen.rmat(9, 16, seed=11, dtype=np.float32)
    full = oracle.spgemm(A, A)
    rows = np.arange(100, 400, dtype=np.int64)
    bound = int(np.minimum(oracle.row_products(A, A, rows), A.ncols).sum())
    one = oracle.spgemm(A, A, rows=rows, capacity=bound)
    two = oracle.spgemm(A, A, rows=rows)
    for f in ("row_ptr", "col_idx", "val", "mag", "products"):
        assert np.array_equal(getattr(one, f), getattr(two, f)), f
    a, b = full.row_ptr[100], full.row_ptr[400]
    assert np.array_equal(one.col_idx, full.col_idx[a:b])
    with pytest.raises(RuntimeError):
        oracle.spgemm(A, A, rows=rows, capacity=two.nnz - 1)


def test_invariants_rmat_small():
    A = matgen.rmat(10, 16, seed=3, dtype=np.float32)
    assert A.is_canonical()
    res = oracle.spgemm(A, A)
    assert_canonical(res, A.nrows, A.ncols)
    nnz_row = np.diff(res.row_ptr)
    assert np.all(nnz_row <= np.minimum(res.products, A.ncols))
    assert np.all((nnz_row == 0) == (res.products == 0))
    # all values positive (inputs in (0, 1]) so M equals the value up to rounding
    assert np.all(res.val > 0)
    assert np.allclose(res.val, res.mag, rtol=1e-6)


def test_check_csr_rejects_noncanonical():
    good = matgen.random_sparse(5, 6, 0.5, 61)
    assert oracle.check_csr(good) == 0
    bad = CSR(good.nrows, good.ncols, good.row_ptr.copy(), good.col_idx.copy(), good.val)
    r = int(np.argmax(np.diff(good.row_ptr) >= 2))
    a = good.row_ptr[r]
    bad.col_idx[a], bad.col_idx[a + 1] = bad.col_idx[a + 1], bad.col_idx[a]
    assert oracle.check_csr(bad) == -4
    bad2 = CSR(good.nrows, 2, good.row_ptr, good.col_idx, good.val)
    assert oracle.check_csr(bad2) == -3
    rp = good.row_ptr.copy()
    rp[0] = 1
    assert oracle.check_csr(CSR(good.nrows, good.ncols, rp, good.col_idx, good.val)) == -2
