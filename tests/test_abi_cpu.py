"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every function include/wingspan.h declares, the workspace size is a
pure function of the sizes, and invalid arguments are rejected with the
documented status codes before any HIP call is made."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_20855_amd import wingspan as ws

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wingspan.h")
FAKE = 0x10000   # a non-null, 256-aligned address that is never dereferenced


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wingspan_\w+)\s*\(", text)))


def desc(nrows, ncols, nnz, rp=FAKE, col=FAKE, val=FAKE):
    d = ws.wingspan_csr()
    d.nrows, d.ncols, d.nnz = nrows, ncols, nnz
    d.row_ptr, d.col_idx, d.val = rp, col, val
    return d


def status_of(fn, *args, **kw):
    with pytest.raises(ws.WingspanError) as e:
        fn(*args, **kw)
    return ws.STATUS[e.value.status], e.value.message


def test_library_exports_every_header_function():
    lib = ws.load()
    declared = header_functions()
    assert set(declared) == set(ws.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_abi_version():
    assert ws.wingspan_abi_version() == ws.ABI_VERSION == 5


def test_struct_layouts_match_header():
    # sizes the C side sees (x86-64 SysV)
    assert ctypes.sizeof(ws.wingspan_csr) == 48
    assert ctypes.sizeof(ws.wingspan_options) == 40
    assert ctypes.sizeof(ws.wingspan_phase_stats) == 4 * 8 * 4 + 4 * 4 + 4 * 4 + 4 + 4 + 8 + 8 + 8


def test_workspace_size_is_host_only_and_monotone():
    small = ws.wingspan_spgemm_workspace_size(desc(1000, 1000, 10_000), desc(1000, 1000, 10_000), ws.F64)
    big = ws.wingspan_spgemm_workspace_size(desc(100_000, 100_000, 1_000_000), desc(100_000, 100_000, 1_000_000),
                                            ws.F64)
    assert 0 < small < big
    assert small % 256 == 0
    # no dense tier -> smaller workspace
    nodense = ws.wingspan_spgemm_workspace_size(desc(100_000, 100_000, 1_000_000),
                                                desc(100_000, 100_000, 1_000_000), ws.F64,
                                                ws.make_options(dense_min_nnz=-1))
    assert nodense < big
    # empty operands are fine, including a B without columns (no structure
    # cache then: its row size would be zero)
    assert ws.wingspan_spgemm_workspace_size(desc(0, 0, 0), desc(0, 0, 0), ws.F32) > 0
    for m, k, n in [(5, 3, 0), (0, 3, 5), (5, 0, 5), (3, 3, 3)]:
        assert ws.wingspan_spgemm_workspace_size(desc(m, k, 0), desc(k, n, 0), ws.F32) > 0


def test_workspace_structure_cache_is_bounded():
    # the dense rows' bitmaps kept from symbolic to numeric take at most 4 GiB, plus two per-row tables (each
    # row's cache slot, and the row order of the numeric binning the symbolic phase keeps)
    n = 262_144
    with_cache = ws.wingspan_spgemm_workspace_size(desc(n, n, 4_000_000), desc(n, n, 4_000_000), ws.F32)
    without = ws.wingspan_spgemm_workspace_size(desc(n, n, 4_000_000), desc(n, n, 4_000_000), ws.F32,
                                                ws.make_options(window_cols=8192))
    assert 0 < with_cache - without <= (4 << 30) + 2 * n * 4 + 1024


def test_workspace_follows_the_cache_budget():
    # options.cache_mib bounds the structure cache: one bitmap of ceil(ncols / 2048) * 256 bytes per row, at most
    # one per row of A; -1 keeps no cache (nor its two per-row tables)
    n = 262_144
    A = B = desc(n, n, 4_000_000)
    row = -(-n // 2048) * 256

    def size(**kw):
        return ws.wingspan_spgemm_workspace_size(A, B, ws.F32, ws.make_options(**kw) if kw else None)

    default = size()
    assert size(cache_mib=4096) == default
    assert default - size(cache_mib=-1) == (4 << 30) // row * row + 2 * n * 4
    # twice the budget caches every row (n rows of 32 KiB each: 8 GiB)
    assert size(cache_mib=8192) - default == (n - (4 << 30) // row) * row
    assert size(cache_mib=16384) == size(cache_mib=8192)
    assert size(cache_mib=1) - size(cache_mib=-1) == (1 << 20) // row * row + 2 * n * 4


@pytest.mark.parametrize("A,B,code", [
    (desc(10, 5, 3), desc(6, 4, 3), "WINGSPAN_ERR_DIMENSION_MISMATCH"),
    (desc(-1, 5, 3), desc(5, 4, 3), "WINGSPAN_ERR_INVALID_ARGUMENT"),
    (desc(10, 5, -3), desc(5, 4, 3), "WINGSPAN_ERR_INVALID_ARGUMENT"),
    (desc(10, 5, 2**31), desc(5, 4, 3), "WINGSPAN_ERR_INDEX_OVERFLOW"),
    (desc(2**31, 5, 3), desc(5, 4, 3), "WINGSPAN_ERR_INDEX_OVERFLOW"),
    (desc(10, 5, 3), desc(5, 2**31, 3), "WINGSPAN_ERR_INDEX_OVERFLOW"),
    (desc(10, 5, 3, rp=0), desc(5, 4, 3), "WINGSPAN_ERR_INVALID_ARGUMENT"),
    (desc(10, 5, 3, col=0), desc(5, 4, 3), "WINGSPAN_ERR_INVALID_ARGUMENT"),
    (desc(10, 5, 3), desc(5, 4, 3, val=0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
])
def test_descriptor_errors(A, B, code):
    got, msg = status_of(ws.wingspan_spgemm_workspace_size, A, B, ws.F64)
    assert got == code and msg
    got2, _ = status_of(ws.wingspan_spgemm_symbolic, A, B, FAKE, FAKE, 1 << 40, 0)
    assert got2 == code
    got3, _ = status_of(ws.wingspan_spgemm_numeric, A, B, ws.F64, FAKE, FAKE, FAKE, FAKE, 1 << 40, 0)
    assert got3 == code
    got4, _ = status_of(ws.wingspan_spgemm_sharded, A, B, ws.F64, FAKE, FAKE, FAKE, FAKE, 10, FAKE, 1 << 40, 0)
    assert got4 == code


def test_null_nnz_zero_pointers_allowed():
    # nnz == 0 matrices may pass NULL col/val
    n = ws.wingspan_spgemm_workspace_size(desc(4, 4, 0, col=0, val=0), desc(4, 4, 0, col=0, val=0), ws.F32)
    assert n > 0


def test_bad_dtype():
    got, _ = status_of(ws.wingspan_spgemm_workspace_size, desc(4, 4, 1), desc(4, 4, 1), 7)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    got, _ = status_of(ws.wingspan_spgemm_numeric, desc(4, 4, 1), desc(4, 4, 1), 2, FAKE, FAKE, FAKE, FAKE,
                       1 << 40, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"


@pytest.mark.parametrize("opts", [
    dict(max_lds_slots=100), dict(max_lds_slots=32), dict(max_lds_slots=1 << 15),
    dict(window_cols=2048), dict(tiny_max=7), dict(tiny_max=65), dict(dense_min_nnz=-2), dict(cache_mib=-2),
])
def test_bad_options(opts):
    got, msg = status_of(ws.wingspan_spgemm_workspace_size, desc(4, 4, 1), desc(4, 4, 1), ws.F32,
                         ws.make_options(**opts))
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT" and "options" in msg


def test_bad_options_version():
    o = ws.make_options()
    o.version = 99
    got, msg = status_of(ws.wingspan_spgemm_workspace_size, desc(4, 4, 1), desc(4, 4, 1), ws.F32, o)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT" and "version" in msg


def test_workspace_too_small_and_misaligned():
    A, B = desc(100, 100, 500), desc(100, 100, 500)
    need = ws.wingspan_spgemm_workspace_size(A, B, ws.F64)
    got, msg = status_of(ws.wingspan_spgemm_symbolic, A, B, FAKE, FAKE, need - 1, 0)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL" and str(need) in msg
    got, _ = status_of(ws.wingspan_spgemm_numeric, A, B, ws.F64, FAKE, FAKE, FAKE, FAKE, need - 256, 0)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"
    got, _ = status_of(ws.wingspan_spgemm_symbolic, A, B, FAKE, FAKE + 8, need, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    got, _ = status_of(ws.wingspan_spgemm_symbolic, A, B, FAKE, 0, need, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"


def test_null_outputs():
    A, B = desc(10, 10, 5), desc(10, 10, 5)
    got, _ = status_of(ws.wingspan_spgemm_symbolic, A, B, 0, FAKE, 1 << 40, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    got, _ = status_of(ws.wingspan_spgemm_numeric, A, B, ws.F64, 0, FAKE, FAKE, FAKE, 1 << 40, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    got, _ = status_of(ws.wingspan_spgemm, A, B, ws.F64, FAKE, FAKE, FAKE, -1, FAKE, 1 << 40, 0)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"


@pytest.mark.parametrize("phase", [-1, 3])
def test_last_stats_bad_phase(phase):
    got, _ = status_of(ws.wingspan_last_stats, phase)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"


def test_error_message_is_thread_local_and_cleared():
    with pytest.raises(ws.WingspanError):
        ws.wingspan_spgemm_workspace_size(desc(3, 4, 1), desc(5, 4, 1), ws.F32)
    assert "A.ncols" in ws.wingspan_last_error()
    ws.wingspan_spgemm_workspace_size(desc(3, 4, 1), desc(4, 4, 1), ws.F32)
    assert ws.wingspan_last_error() == ""


def sharded(A, B, dtype=None, row_off=FAKE, row_nnz=FAKE, pool_col=FAKE, pool_val=FAKE, cap=10, wsp=FAKE,
            wsb=1 << 40, options=None):
    return ws.wingspan_spgemm_sharded(A, B, ws.F64 if dtype is None else dtype, row_off, row_nnz, pool_col,
                                      pool_val, cap, wsp, wsb, 0, options)


def test_sharded_argument_errors():
    A, B = desc(10, 10, 5), desc(10, 10, 5)
    for kw in [dict(dtype=3), dict(cap=-1), dict(row_off=0), dict(row_nnz=0), dict(pool_col=0), dict(pool_val=0),
               dict(wsp=0), dict(wsp=FAKE + 8)]:
        got, msg = status_of(sharded, A, B, **kw)
        assert got == "WINGSPAN_ERR_INVALID_ARGUMENT" and msg, kw
    need = ws.wingspan_spgemm_workspace_size(A, B, ws.F64)
    got, msg = status_of(sharded, A, B, wsb=need - 1)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL" and str(need) in msg
    got, _ = status_of(sharded, A, B, options=ws.make_options(max_lds_slots=100))
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    # an empty pool may be NULL (the call then only counts); empty A may pass NULL row arrays: these get past
    # the argument checks and stop at the workspace check
    got, _ = status_of(sharded, A, B, pool_col=0, pool_val=0, cap=0, wsb=need - 1)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"
    E = desc(0, 10, 0, col=0, val=0)
    got, _ = status_of(sharded, E, B, row_off=0, row_nnz=0, wsb=0)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"


def test_sharded_to_csr_workspace_and_errors():
    sizes = [ws.wingspan_sharded_to_csr_workspace_size(n) for n in (0, 1, 1000, 10 ** 6)]
    assert all(b > 0 and b % 256 == 0 for b in sizes) and sizes == sorted(sizes)
    got, _ = status_of(ws.wingspan_sharded_to_csr_workspace_size, -1)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    need = ws.wingspan_sharded_to_csr_workspace_size(10)
    args = dict(nrows=10, nnz=5, row_off=FAKE, row_nnz=FAKE, pool_col=FAKE, pool_val=FAKE, dtype=ws.F32,
                c_row_ptr=FAKE, c_col_idx=FAKE, c_val=FAKE, workspace=FAKE, workspace_bytes=need)
    for kw, code in [(dict(dtype=5), "WINGSPAN_ERR_INVALID_ARGUMENT"), (dict(c_row_ptr=0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                     (dict(row_off=0), "WINGSPAN_ERR_INVALID_ARGUMENT"), (dict(nrows=-3), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                     (dict(nnz=-1), "WINGSPAN_ERR_INVALID_ARGUMENT"), (dict(pool_col=0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                     (dict(c_val=0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                     (dict(workspace_bytes=need - 1), "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"),
                     (dict(workspace=FAKE + 8), "WINGSPAN_ERR_INVALID_ARGUMENT")]:
        got, _ = status_of(ws.wingspan_sharded_to_csr, **{**args, **kw})
        assert got == code, kw


def test_elementwise_argument_errors():
    A, B = desc(10, 12, 5), desc(10, 12, 7)
    need = ws.wingspan_elementwise_workspace_size(A, B)
    assert need > 0 and need % 256 == 0
    assert ws.wingspan_elementwise_workspace_size(desc(10, 12, 5_000_000), B) > need   # one boundary per 2048 entries
    got, _ = status_of(ws.wingspan_elementwise_workspace_size, A, desc(10, 13, 7))
    assert got == "WINGSPAN_ERR_DIMENSION_MISMATCH"
    got, _ = status_of(ws.wingspan_elementwise_structure, ws.OP_ADD, A, desc(11, 12, 7), FAKE, FAKE, need, 0)
    assert got == "WINGSPAN_ERR_DIMENSION_MISMATCH"
    for args, code in [((5, A, B, FAKE, FAKE, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_ADD, A, B, 0, FAKE, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_ADD, A, B, FAKE, FAKE, need - 1, 0), "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"),
                       ((ws.OP_HADAMARD, A, B, FAKE, 0, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_HADAMARD, A, B, FAKE, FAKE + 8, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT")]:
        got, _ = status_of(ws.wingspan_elementwise_structure, *args)
        assert got == code, args
    for args, code in [((ws.OP_ADD, A, B, 9, FAKE, FAKE, FAKE, FAKE, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_ADD, A, B, ws.F32, FAKE, 0, FAKE, FAKE, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_ADD, A, B, ws.F32, 0, FAKE, FAKE, FAKE, need, 0), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((ws.OP_HADAMARD, A, B, ws.F64, FAKE, FAKE, FAKE, FAKE, need - 256, 0),
                        "WINGSPAN_ERR_WORKSPACE_TOO_SMALL")]:
        got, _ = status_of(ws.wingspan_elementwise_values, *args)
        assert got == code, args


def test_spmspv_argument_errors():
    At = desc(12, 10, 30)   # A is 10 x 12, given by its 12 columns
    need = ws.wingspan_spmspv_workspace_size(At, 5)
    assert need > 0 and need % 256 == 0
    assert ws.wingspan_spmspv_workspace_size(desc(12, 100000, 30), 5) > need
    for args in [(At, -1), (At, 13), (desc(12, 10, -1), 5)]:
        got, _ = status_of(ws.wingspan_spmspv_workspace_size, *args)
        assert got == "WINGSPAN_ERR_INVALID_ARGUMENT", args
    for args, code in [((At, 9, FAKE, FAKE, 5, FAKE, FAKE, 10, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F32, 0, FAKE, 5, FAKE, FAKE, 10, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F32, FAKE, 0, 5, FAKE, FAKE, 10, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F32, FAKE, FAKE, 5, FAKE, FAKE, -1, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F32, FAKE, FAKE, 5, 0, FAKE, 10, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F64, FAKE, FAKE, 5, FAKE, FAKE, 10, FAKE, need - 1),
                        "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"),
                       ((At, ws.F64, FAKE, FAKE, 5, FAKE, FAKE, 10, 0, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F64, FAKE, FAKE, 5, FAKE, FAKE, 10, FAKE + 8, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, ws.F64, FAKE, FAKE, 13, FAKE, FAKE, 10, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((desc(2**31, 10, 3), ws.F64, FAKE, FAKE, 1, FAKE, FAKE, 10, FAKE, need),
                        "WINGSPAN_ERR_INDEX_OVERFLOW")]:
        got, _ = status_of(ws.wingspan_spmspv, *args)
        assert got == code, args
    lib = ws.load()
    st = lib.wingspan_spmspv(ctypes.byref(At), ws.F32, FAKE, FAKE, 5, FAKE, FAKE, 10, None, FAKE, need, None)
    assert ws.STATUS[st] == "WINGSPAN_ERR_INVALID_ARGUMENT"


def test_outer_argument_errors():
    At, B = desc(9, 12, 30), desc(9, 15, 40)   # A is 12 x 9 (by its 9 columns), B is 9 x 15
    base = ws.wingspan_outer_workspace_size(At, B, 0)
    full = ws.wingspan_outer_workspace_size(At, B, 100000)
    assert base % 256 == 0 and full > base
    got, _ = status_of(ws.wingspan_outer_workspace_size, At, desc(10, 15, 40), 0)
    assert got == "WINGSPAN_ERR_DIMENSION_MISMATCH"
    got, _ = status_of(ws.wingspan_outer_workspace_size, At, B, -1)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    got, _ = status_of(ws.wingspan_outer_products, At, B, FAKE, 0)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"
    got, _ = status_of(ws.wingspan_outer_products, At, B, FAKE + 8, base)
    assert got == "WINGSPAN_ERR_INVALID_ARGUMENT"
    for args, code in [((At, B, 9, FAKE, FAKE, FAKE, 10, FAKE, full), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, B, ws.F32, 0, FAKE, FAKE, 10, FAKE, full), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, B, ws.F32, FAKE, 0, FAKE, 10, FAKE, full), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, B, ws.F32, FAKE, FAKE, FAKE, -1, FAKE, full), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, B, ws.F64, FAKE, FAKE, FAKE, 10, 0, full), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((At, B, ws.F64, FAKE, FAKE, FAKE, 10, FAKE, 16), "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"),
                       ((At, desc(9, 15, -2), ws.F64, FAKE, FAKE, FAKE, 10, FAKE, full), "WINGSPAN_ERR_INVALID_ARGUMENT")]:
        got, _ = status_of(ws.wingspan_spgemm_outer, *args)
        assert got == code, args


def test_row_products_argument_errors():
    A, B = desc(10, 12, 5), desc(12, 7, 9)
    need = ws.wingspan_spgemm_workspace_size(A, B, ws.F64)
    got, _ = status_of(ws.wingspan_spgemm_row_products, A, desc(11, 7, 9), FAKE, FAKE, need)
    assert got == "WINGSPAN_ERR_DIMENSION_MISMATCH"
    for args, code in [((A, B, 0, FAKE, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((A, B, FAKE, FAKE, need - 1), "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"),
                       ((A, B, FAKE, 0, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((A, B, FAKE, FAKE + 8, need), "WINGSPAN_ERR_INVALID_ARGUMENT"),
                       ((desc(10, 12, 2**31), B, FAKE, FAKE, need), "WINGSPAN_ERR_INDEX_OVERFLOW")]:
        got, _ = status_of(ws.wingspan_spgemm_row_products, *args)
        assert got == code, args
    # an A without rows may pass a NULL output (it then stops at the workspace check)
    got, _ = status_of(ws.wingspan_spgemm_row_products, desc(0, 12, 0, col=0, val=0), B, 0, FAKE, 0)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL"


def test_noalloc_argument_errors():
    A, B = desc(10, 12, 5), desc(12, 7, 9)
    call = ws.wingspan_spgemm_noalloc
    for args, kw, code in [((A, desc(11, 7, 9), ws.F64, FAKE, FAKE, FAKE, 10), {}, "WINGSPAN_ERR_DIMENSION_MISMATCH"),
                           ((A, B, 7, FAKE, FAKE, FAKE, 10), {}, "WINGSPAN_ERR_INVALID_ARGUMENT"),
                           ((A, B, ws.F64, 0, FAKE, FAKE, 10), {}, "WINGSPAN_ERR_INVALID_ARGUMENT"),
                           ((A, B, ws.F64, FAKE, FAKE, FAKE, -1), {}, "WINGSPAN_ERR_INVALID_ARGUMENT"),
                           ((A, B, ws.F64, FAKE, FAKE, FAKE, 10), dict(options=ws.make_options(timing=1)),
                            "WINGSPAN_ERR_INVALID_ARGUMENT"),
                           ((A, B, ws.F64, FAKE, FAKE, FAKE, 10), dict(options=ws.make_options(max_lds_slots=100)),
                            "WINGSPAN_ERR_INVALID_ARGUMENT")]:
        got, _ = status_of(call, *args, **kw)
        assert got == code, (args, kw)
    # a product whose scratch would pass the static array's size is refused before any HIP call
    big = desc(2**30, 2**30, 2**31 - 1)
    got, msg = status_of(call, big, big, ws.F32, FAKE, FAKE, FAKE, 10)
    assert got == "WINGSPAN_ERR_WORKSPACE_TOO_SMALL" and str(ws.NOALLOC_SCRATCH_BYTES) in msg
    lib = ws.load()
    st = lib.wingspan_spgemm_noalloc(ctypes.byref(A), ctypes.byref(B), ws.F64, FAKE, FAKE, FAKE, 10, None, None,
                                     None)
    assert ws.STATUS[st] == "WINGSPAN_ERR_INVALID_ARGUMENT"
