"""The numeric phase's reuse of the column sets that the symbolic phase leaves
in the workspace (the structure cache): taken when the workspace's stamp
matches the numeric call, ignored otherwise, and the result equals the
oracle's either way."""
from __future__ import annotations

import numpy as np
import pytest

import matgen
import oracle
from gpu_util import assert_matches

pytestmark = pytest.mark.gpu

# rows above 42 output entries skip the LDS hash tiers: many dense rows on
# R-MAT scale 11
DENSE = dict(tiny_max=-1, max_lds_slots=64)


def _dev(A):
    from paper_2606_20855_amd import wingspan as ws
    return ws.DeviceCSR.from_host(A, "cuda:0")


def _symbolic(dA, dB, wsb, nbytes, opts):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    c_rp = torch.empty(dA.nrows + 1, dtype=torch.int64, device="cuda:0")
    nnz = ws.wingspan_spgemm_symbolic(dA.desc(), dB.desc(), c_rp.data_ptr(), wsb.data_ptr(), nbytes, None,
                                      ws.make_options(**opts))
    return c_rp, nnz


def _numeric(dA, dB, c_rp, nnz, wsb, nbytes, opts):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    c_col = torch.empty(max(nnz, 1), dtype=torch.int32, device="cuda:0")
    c_val = torch.empty(max(nnz, 1), dtype=dA.val.dtype, device="cuda:0")
    ws.wingspan_spgemm_numeric(dA.desc(), dB.desc(), dA.dtype_code, c_rp.data_ptr(), c_col.data_ptr(),
                               c_val.data_ptr(), wsb.data_ptr(), nbytes, None, ws.make_options(**opts))
    torch.cuda.synchronize()
    C = ws.DeviceCSR(dA.nrows, dB.ncols, c_rp, c_col[:nnz], c_val[:nnz]).to_host()
    return C, ws.wingspan_last_stats(1)


def _workspace(dA, dB, opts):
    import torch
    from paper_2606_20855_amd import wingspan as ws
    nbytes = ws.wingspan_spgemm_workspace_size(dA.desc(), dB.desc(), dA.dtype_code, ws.make_options(**opts))
    # zero-filled: a fresh workspace holds no valid stamp
    return torch.zeros(nbytes, dtype=torch.uint8, device="cuda:0"), nbytes


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_cache_used_after_symbolic(dtype):
    A = matgen.rmat(11, 16, seed=51, dtype=dtype, dist="open01" if dtype == np.float32 else "pm1")
    dA = _dev(A)
    wsb, nbytes = _workspace(dA, dA, DENSE)
    c_rp, nnz = _symbolic(dA, dA, wsb, nbytes, DENSE)
    got, num = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, DENSE)
    assert num["rows"]["dense"] > 0
    assert num["structure_cache_rows"] > 0
    assert_matches(got, oracle.spgemm(A, A), A.val.dtype, what="cache used")
    # a second numeric call on the same workspace reuses it again
    got2, num2 = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, DENSE)
    assert num2["structure_cache_rows"] == num["structure_cache_rows"]
    assert np.array_equal(got2.col_idx, got.col_idx)


def test_fresh_workspace_recomputes():
    A = matgen.rmat(11, 16, seed=52, dtype=np.float32)
    dA = _dev(A)
    ws1, nbytes = _workspace(dA, dA, DENSE)
    ws2, _ = _workspace(dA, dA, DENSE)
    c_rp, nnz = _symbolic(dA, dA, ws1, nbytes, DENSE)
    got, num = _numeric(dA, dA, c_rp, nnz, ws2, nbytes, DENSE)
    assert num["rows"]["dense"] > 0 and num["structure_cache_rows"] == 0
    assert_matches(got, oracle.spgemm(A, A), A.val.dtype, what="fresh workspace")


def test_stamp_of_another_pair_is_ignored():
    A1 = matgen.rmat(11, 16, seed=53, dtype=np.float32)
    A2 = matgen.rmat(11, 16, seed=54, dtype=np.float32)
    import torch
    from paper_2606_20855_amd import wingspan as ws
    d1, d2 = _dev(A1), _dev(A2)
    nbytes = max(ws.wingspan_spgemm_workspace_size(d.desc(), d.desc(), d.dtype_code, ws.make_options(**DENSE))
                 for d in (d1, d2))
    wsb = torch.zeros(nbytes, dtype=torch.uint8, device="cuda:0")
    rp1, nnz1 = _symbolic(d1, d1, wsb, nbytes, DENSE)
    _symbolic(d2, d2, wsb, nbytes, DENSE)          # leaves A2's stamp in the workspace
    got, num = _numeric(d1, d1, rp1, nnz1, wsb, nbytes, DENSE)
    assert num["structure_cache_rows"] == 0
    assert_matches(got, oracle.spgemm(A1, A1), A1.val.dtype, what="other stamp")


def test_pattern_changed_in_place_is_detected_by_row_ptr():
    # same buffers and sizes, new pattern (columns permuted): only the C.row_ptr
    # checksum tells the stale cache apart
    import torch
    A1 = matgen.rmat(11, 16, seed=55, dtype=np.float32)
    perm = np.random.default_rng(7).permutation(A1.ncols).astype(np.int32)
    cols = perm[A1.col_idx]
    rows = np.repeat(np.arange(A1.nrows), np.diff(A1.row_ptr))
    order = np.lexsort((cols, rows))
    A2 = matgen.CSR(A1.nrows, A1.ncols, A1.row_ptr.copy(), cols[order].astype(np.int32), A1.val[order].copy())
    assert A2.is_canonical()
    d = _dev(A1)
    wsb, nbytes = _workspace(d, d, DENSE)
    rp1, _ = _symbolic(d, d, wsb, nbytes, DENSE)
    d.col_idx.copy_(torch.from_numpy(A2.col_idx).to("cuda:0"))
    d.val.copy_(torch.from_numpy(A2.val).to("cuda:0"))
    other, _ = _workspace(d, d, DENSE)
    rp2, nnz2 = _symbolic(d, d, other, nbytes, DENSE)
    if torch.equal(rp1, rp2):
        pytest.skip("the permuted pattern happens to give the same C.row_ptr")
    got, num = _numeric(d, d, rp2, nnz2, wsb, nbytes, DENSE)
    assert num["structure_cache_rows"] == 0
    assert_matches(got, oracle.spgemm(A2, A2), A2.val.dtype, what="pattern changed")


def test_other_layout_recomputes():
    A = matgen.rmat(11, 16, seed=56, dtype=np.float32)
    dA = _dev(A)
    other = dict(DENSE, window_cols=1024)   # column-window kernel, no cache
    import torch
    from paper_2606_20855_amd import wingspan as ws
    nbytes = max(ws.wingspan_spgemm_workspace_size(dA.desc(), dA.desc(), dA.dtype_code, ws.make_options(**o))
                 for o in (DENSE, other))
    wsb = torch.zeros(nbytes, dtype=torch.uint8, device="cuda:0")
    c_rp, nnz = _symbolic(dA, dA, wsb, nbytes, DENSE)
    got, num = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, other)
    assert num["structure_cache_rows"] == 0
    assert_matches(got, oracle.spgemm(A, A), A.val.dtype, what="other layout")


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_long_rows_cached_and_fresh(dtype):
    # rows with more A entries than the rank kernel keeps in LDS, several rank
    # slices and two 262144-column regions: the cached bitmap and the
    # structure pass give the same C
    dist = "open01" if dtype == np.float32 else "pm1"
    A = matgen.er(24, 2500, 300, seed=57, dtype=dtype, dist=dist)
    B = matgen.er(2500, 280_000, 40, seed=58, dtype=dtype, dist=dist)
    dA, dB = _dev(A), _dev(B)
    wsb, nbytes = _workspace(dA, dB, {})
    fresh, _ = _workspace(dA, dB, {})
    c_rp, nnz = _symbolic(dA, dB, wsb, nbytes, {})
    got, num = _numeric(dA, dB, c_rp, nnz, wsb, nbytes, {})
    assert num["rows"]["dense"] == 24 and num["structure_cache_rows"] == 24
    ref = oracle.spgemm(A, B)
    assert_matches(got, ref, A.val.dtype, what="long rows, cached")
    got2, num2 = _numeric(dA, dB, c_rp, nnz, fresh, nbytes, {})
    assert num2["structure_cache_rows"] == 0
    assert_matches(got2, ref, A.val.dtype, what="long rows, fresh")


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_wide_offsets_path(dtype):
    # the rank kernel forms B's offsets in 32 bits unless nnz(B) * sizeof(value) exceeds 2^32; the switch
    # takes the 64-bit path on a small B, which must give the same C
    A = matgen.rmat(11, 16, seed=59, dtype=dtype, dist="open01" if dtype == np.float32 else "pm1")
    dA = _dev(A)
    ref = oracle.spgemm(A, A)
    for opts in (DENSE, dict(DENSE, wide_offsets=1)):
        wsb, nbytes = _workspace(dA, dA, opts)
        c_rp, nnz = _symbolic(dA, dA, wsb, nbytes, opts)
        got, num = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, opts)
        assert num["rows"]["dense"] > 0
        assert_matches(got, ref, A.val.dtype, what=f"offsets {opts}")


@pytest.mark.parametrize("change", [dict(tiny_max=16), dict(max_lds_slots=512), dict(dense_min_nnz=200),
                                    dict(force_spill=1)])
def test_numeric_settings_differ_from_symbolic(change):
    # the symbolic phase bins the rows for a numeric phase with its own settings; a numeric call with other
    # settings (same layout) must bin them itself, and match the oracle
    A = matgen.rmat(11, 16, seed=61, dtype=np.float32)
    dA = _dev(A)
    ref = oracle.spgemm(A, A)
    wsb, nbytes = _workspace(dA, dA, DENSE)
    c_rp, nnz = _symbolic(dA, dA, wsb, nbytes, DENSE)
    got, num = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, dict(DENSE, **change))
    assert_matches(got, ref, A.val.dtype, what=f"numeric {change}")
    if change.get("force_spill"):
        assert num["rows"]["spill"] > 0 and num["rows"]["dense"] == 0
    # and the same workspace again with the symbolic phase's own settings
    got2, num2 = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, DENSE)
    assert_matches(got2, ref, A.val.dtype, what="numeric with the symbolic settings")
    assert num2["structure_cache_rows"] > 0 and num2["rows"]["dense"] > 0


def test_single_pass_between_phases_invalidates_the_kept_state():
    # the single pass (sharded output) reuses the workspace's row tables; a numeric phase after it on the same
    # workspace must not take the symbolic phase's kept state, and still matches the oracle
    from paper_2606_20855_amd import wingspan as ws
    A = matgen.rmat(11, 16, seed=63, dtype=np.float32)
    dA = _dev(A)
    ref = oracle.spgemm(A, A)
    wsb, nbytes = _workspace(dA, dA, DENSE)
    c_rp, nnz = _symbolic(dA, dA, wsb, nbytes, DENSE)
    S = ws.spgemm_sharded(dA, dA, options=ws.make_options(**DENSE), workspace=wsb)
    assert S.nnz == nnz
    got, num = _numeric(dA, dA, c_rp, nnz, wsb, nbytes, DENSE)
    assert num["structure_cache_rows"] == 0
    assert_matches(got, ref, A.val.dtype, what="numeric after a single pass")


@pytest.mark.parametrize("cache_mib,cached", [(-1, 0), (1, 8), (0, 64)])
def test_cache_budget_bounds_the_cached_rows(cache_mib, cached):
    # B has 2^20 columns, so a row's bitmap takes 128 KiB: 1 MiB holds 8 of the 64 dense rows, the default
    # budget all of them, -1 none; the rows past the budget run their own structure pass
    A = matgen.er(64, 512, 16, seed=57, dtype=np.float32, dist="open01")
    B = matgen.er(512, 1 << 20, 64, seed=58, dtype=np.float32, dist="open01")
    opts = dict(DENSE, cache_mib=cache_mib)
    dA, dB = _dev(A), _dev(B)
    wsb, nbytes = _workspace(dA, dB, opts)
    c_rp, nnz = _symbolic(dA, dB, wsb, nbytes, opts)
    got, num = _numeric(dA, dB, c_rp, nnz, wsb, nbytes, opts)
    assert num["rows"]["dense"] == 64
    assert num["structure_cache_rows"] == cached
    assert_matches(got, oracle.spgemm(A, B), A.val.dtype, what=f"cache budget {cache_mib} MiB")
