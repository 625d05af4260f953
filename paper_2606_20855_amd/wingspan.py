"""Python binding of the gfx950 SpGEMM C ABI (include/wingspan.h).

The functions named ``wingspan_*`` mirror the C entry points one to one and
only marshal arguments; all computation happens in libwingspan.so on the GPU.
``spgemm()`` is a convenience wrapper that allocates the workspace and C with
torch (device memory and streams only) and runs both phases.

There is no fallback: if libwingspan.so is missing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libwingspan.so")

ABI_VERSION = 5
F32, F64 = 0, 1
OP_ADD, OP_HADAMARD = 0, 1
TIERS = ("tiny", "hash", "dense", "spill")

STATUS = {
    0: "WINGSPAN_OK",
    1: "WINGSPAN_ERR_INVALID_ARGUMENT",
    2: "WINGSPAN_ERR_DIMENSION_MISMATCH",
    3: "WINGSPAN_ERR_INDEX_OVERFLOW",
    4: "WINGSPAN_ERR_WORKSPACE_TOO_SMALL",
    5: "WINGSPAN_ERR_INSUFFICIENT_CAPACITY",
    6: "WINGSPAN_ERR_INVALID_MATRIX",
    7: "WINGSPAN_ERR_HIP",
    8: "WINGSPAN_ERR_UNSUPPORTED",
    9: "WINGSPAN_ERR_INCONSISTENT",
}
STATUS_CODE = {v: k for k, v in STATUS.items()}


class WingspanError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class wingspan_csr(ctypes.Structure):
    _fields_ = [
        ("nrows", ctypes.c_int64),
        ("ncols", ctypes.c_int64),
        ("nnz", ctypes.c_int64),
        ("row_ptr", ctypes.c_void_p),
        ("col_idx", ctypes.c_void_p),
        ("val", ctypes.c_void_p),
    ]


class wingspan_options(ctypes.Structure):
    _fields_ = [
        ("version", ctypes.c_uint32),
        ("validate", ctypes.c_int32),
        ("max_lds_slots", ctypes.c_int32),
        ("force_spill", ctypes.c_int32),
        ("window_cols", ctypes.c_int32),
        ("tiny_max", ctypes.c_int32),
        ("dense_min_nnz", ctypes.c_int32),
        ("timing", ctypes.c_int32),
        ("wide_offsets", ctypes.c_int32),
        ("cache_mib", ctypes.c_int32),
    ]


_NT = 4


class wingspan_phase_stats(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64 * _NT),
        ("a_nnz", ctypes.c_int64 * _NT),
        ("products", ctypes.c_int64 * _NT),
        ("c_nnz", ctypes.c_int64 * _NT),
        ("launches", ctypes.c_int32 * _NT),
        ("kernel_ms", ctypes.c_float * _NT),
        ("analysis_ms", ctypes.c_float),
        ("total_products", ctypes.c_int64),
        ("c_nnz_total", ctypes.c_int64),
        ("structure_cache_rows", ctypes.c_int64),
    ]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libwingspan.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python __graft_entry__.py build` "
                           "(or paper_2606_20855_amd._build.build())")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    csr_p, opt_p = P(wingspan_csr), P(wingspan_options)
    lib.wingspan_abi_version.argtypes = []
    lib.wingspan_abi_version.restype = i32
    lib.wingspan_last_error.argtypes = []
    lib.wingspan_last_error.restype = ctypes.c_char_p
    lib.wingspan_last_stats.argtypes = [i32, P(wingspan_phase_stats)]
    lib.wingspan_last_stats.restype = i32
    lib.wingspan_spgemm_workspace_size.argtypes = [csr_p, csr_p, i32, opt_p, P(sz)]
    lib.wingspan_spgemm_workspace_size.restype = i32
    lib.wingspan_spgemm_symbolic.argtypes = [csr_p, csr_p, vp, P(i64), vp, sz, vp, opt_p]
    lib.wingspan_spgemm_symbolic.restype = i32
    lib.wingspan_spgemm_numeric.argtypes = [csr_p, csr_p, i32, vp, vp, vp, vp, sz, vp, opt_p]
    lib.wingspan_spgemm_numeric.restype = i32
    lib.wingspan_spgemm.argtypes = [csr_p, csr_p, i32, vp, vp, vp, i64, P(i64), vp, sz, vp, opt_p]
    lib.wingspan_spgemm.restype = i32
    lib.wingspan_spgemm_noalloc.argtypes = [csr_p, csr_p, i32, vp, vp, vp, i64, P(i64), vp, opt_p]
    lib.wingspan_spgemm_noalloc.restype = i32
    lib.wingspan_spgemm_row_products.argtypes = [csr_p, csr_p, vp, vp, sz, vp]
    lib.wingspan_spgemm_row_products.restype = i32
    lib.wingspan_spgemm_sharded.argtypes = [csr_p, csr_p, i32, vp, vp, vp, vp, i64, P(i64), vp, sz, vp, opt_p]
    lib.wingspan_spgemm_sharded.restype = i32
    lib.wingspan_sharded_to_csr_workspace_size.argtypes = [i64, P(sz)]
    lib.wingspan_sharded_to_csr_workspace_size.restype = i32
    lib.wingspan_sharded_to_csr.argtypes = [i64, i64, vp, vp, vp, vp, i32, vp, vp, vp, vp, sz, vp]
    lib.wingspan_sharded_to_csr.restype = i32
    lib.wingspan_elementwise_workspace_size.argtypes = [csr_p, csr_p, P(sz)]
    lib.wingspan_elementwise_workspace_size.restype = i32
    lib.wingspan_elementwise_structure.argtypes = [i32, csr_p, csr_p, vp, P(i64), vp, sz, vp]
    lib.wingspan_elementwise_structure.restype = i32
    lib.wingspan_elementwise_values.argtypes = [i32, csr_p, csr_p, i32, vp, vp, vp, vp, sz, vp]
    lib.wingspan_elementwise_values.restype = i32
    lib.wingspan_spmspv_workspace_size.argtypes = [csr_p, i64, P(sz)]
    lib.wingspan_spmspv_workspace_size.restype = i32
    lib.wingspan_spmspv.argtypes = [csr_p, i32, vp, vp, i64, vp, vp, i64, P(i64), vp, sz, vp]
    lib.wingspan_spmspv.restype = i32
    lib.wingspan_outer_workspace_size.argtypes = [csr_p, csr_p, i64, P(sz)]
    lib.wingspan_outer_workspace_size.restype = i32
    lib.wingspan_outer_products.argtypes = [csr_p, csr_p, P(i64), vp, sz, vp]
    lib.wingspan_outer_products.restype = i32
    lib.wingspan_spgemm_outer.argtypes = [csr_p, csr_p, i32, vp, vp, vp, i64, P(i64), vp, sz, vp]
    lib.wingspan_spgemm_outer.restype = i32
    _lib = lib
    return lib


EXPORTED = (
    "wingspan_abi_version",
    "wingspan_last_error",
    "wingspan_last_stats",
    "wingspan_spgemm_workspace_size",
    "wingspan_spgemm_symbolic",
    "wingspan_spgemm_numeric",
    "wingspan_spgemm",
    "wingspan_spgemm_noalloc",
    "wingspan_spgemm_row_products",
    "wingspan_spgemm_sharded",
    "wingspan_sharded_to_csr_workspace_size",
    "wingspan_sharded_to_csr",
    "wingspan_elementwise_workspace_size",
    "wingspan_elementwise_structure",
    "wingspan_elementwise_values",
    "wingspan_spmspv_workspace_size",
    "wingspan_spmspv",
    "wingspan_outer_workspace_size",
    "wingspan_outer_products",
    "wingspan_spgemm_outer",
)


def make_options(**kw) -> wingspan_options:
    o = wingspan_options()
    o.version = ABI_VERSION
    for k, v in kw.items():
        if not hasattr(o, k) or k == "version":
            raise KeyError(k)
        setattr(o, k, int(v))
    return o


def _opt_ptr(options):
    if options is None:
        return None
    if isinstance(options, dict):
        options = make_options(**options)
    return ctypes.byref(options)


def _check(status: int):
    if status != 0:
        raise WingspanError(status, load().wingspan_last_error().decode())


def wingspan_abi_version() -> int:
    return load().wingspan_abi_version()


def wingspan_last_error() -> str:
    return load().wingspan_last_error().decode()


def wingspan_last_stats(phase: int) -> dict:
    st = wingspan_phase_stats()
    _check(load().wingspan_last_stats(phase, ctypes.byref(st)))
    out = {name: {t: getattr(st, name)[i] for i, t in enumerate(TIERS)}
           for name in ("rows", "a_nnz", "products", "c_nnz", "launches", "kernel_ms")}
    out["analysis_ms"] = st.analysis_ms
    out["total_products"] = st.total_products
    out["c_nnz_total"] = st.c_nnz_total
    out["structure_cache_rows"] = st.structure_cache_rows
    return out


def wingspan_spgemm_workspace_size(A: wingspan_csr, B: wingspan_csr, dtype: int, options=None) -> int:
    n = ctypes.c_size_t(0)
    _check(load().wingspan_spgemm_workspace_size(ctypes.byref(A), ctypes.byref(B), dtype, _opt_ptr(options),
                                                 ctypes.byref(n)))
    return n.value


def wingspan_spgemm_symbolic(A: wingspan_csr, B: wingspan_csr, c_row_ptr: int, workspace: int,
                             workspace_bytes: int, stream: int = 0, options=None) -> int:
    nnz = ctypes.c_int64(0)
    _check(load().wingspan_spgemm_symbolic(ctypes.byref(A), ctypes.byref(B), c_row_ptr, ctypes.byref(nnz),
                                           workspace, workspace_bytes, stream or None, _opt_ptr(options)))
    return nnz.value


def wingspan_spgemm_numeric(A: wingspan_csr, B: wingspan_csr, dtype: int, c_row_ptr: int, c_col_idx: int,
                            c_val: int, workspace: int, workspace_bytes: int, stream: int = 0,
                            options=None) -> None:
    _check(load().wingspan_spgemm_numeric(ctypes.byref(A), ctypes.byref(B), dtype, c_row_ptr, c_col_idx, c_val,
                                          workspace, workspace_bytes, stream or None, _opt_ptr(options)))


def wingspan_spgemm(A: wingspan_csr, B: wingspan_csr, dtype: int, c_row_ptr: int, c_col_idx: int, c_val: int,
                    c_capacity: int, workspace: int, workspace_bytes: int, stream: int = 0,
                    options=None) -> int:
    nnz = ctypes.c_int64(0)
    _check(load().wingspan_spgemm(ctypes.byref(A), ctypes.byref(B), dtype, c_row_ptr, c_col_idx, c_val,
                                  c_capacity, ctypes.byref(nnz), workspace, workspace_bytes, stream or None,
                                  _opt_ptr(options)))
    return nnz.value


NOALLOC_SCRATCH_BYTES = 256 << 20   # WINGSPAN_NOALLOC_SCRATCH_BYTES


def wingspan_spgemm_noalloc(A: wingspan_csr, B: wingspan_csr, dtype: int, c_row_ptr: int, c_col_idx: int,
                            c_val: int, c_capacity: int, stream: int = 0, options=None) -> int:
    nnz = ctypes.c_int64(0)
    _check(load().wingspan_spgemm_noalloc(ctypes.byref(A), ctypes.byref(B), dtype, c_row_ptr, c_col_idx or None,
                                          c_val or None, c_capacity, ctypes.byref(nnz), stream or None,
                                          _opt_ptr(options)))
    return nnz.value


def wingspan_spgemm_row_products(A: wingspan_csr, B: wingspan_csr, row_products: int, workspace: int,
                                 workspace_bytes: int, stream: int = 0) -> None:
    _check(load().wingspan_spgemm_row_products(ctypes.byref(A), ctypes.byref(B), row_products or None, workspace,
                                               workspace_bytes, stream or None))


def wingspan_spgemm_sharded(A: wingspan_csr, B: wingspan_csr, dtype: int, row_off: int, row_nnz: int,
                            pool_col: int, pool_val: int, pool_capacity: int, workspace: int,
                            workspace_bytes: int, stream: int = 0, options=None, check: bool = True):
    """Returns (status, pool_used). With check=True a non-OK status raises."""
    used = ctypes.c_int64(0)
    st = load().wingspan_spgemm_sharded(ctypes.byref(A), ctypes.byref(B), dtype, row_off, row_nnz, pool_col,
                                        pool_val, pool_capacity, ctypes.byref(used), workspace, workspace_bytes,
                                        stream or None, _opt_ptr(options))
    if check:
        _check(st)
    return st, used.value


def wingspan_sharded_to_csr_workspace_size(nrows: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().wingspan_sharded_to_csr_workspace_size(nrows, ctypes.byref(n)))
    return n.value


def wingspan_sharded_to_csr(nrows: int, nnz: int, row_off: int, row_nnz: int, pool_col: int, pool_val: int,
                            dtype: int, c_row_ptr: int, c_col_idx: int, c_val: int, workspace: int,
                            workspace_bytes: int, stream: int = 0) -> None:
    _check(load().wingspan_sharded_to_csr(nrows, nnz, row_off, row_nnz, pool_col, pool_val, dtype, c_row_ptr,
                                          c_col_idx, c_val, workspace, workspace_bytes, stream or None))


def wingspan_elementwise_workspace_size(A: wingspan_csr, B: wingspan_csr) -> int:
    n = ctypes.c_size_t(0)
    _check(load().wingspan_elementwise_workspace_size(ctypes.byref(A), ctypes.byref(B), ctypes.byref(n)))
    return n.value


def wingspan_elementwise_structure(op: int, A: wingspan_csr, B: wingspan_csr, c_row_ptr: int, workspace: int,
                                   workspace_bytes: int, stream: int = 0) -> int:
    nnz = ctypes.c_int64(0)
    _check(load().wingspan_elementwise_structure(op, ctypes.byref(A), ctypes.byref(B), c_row_ptr, ctypes.byref(nnz),
                                                 workspace, workspace_bytes, stream or None))
    return nnz.value


def wingspan_elementwise_values(op: int, A: wingspan_csr, B: wingspan_csr, dtype: int, c_row_ptr: int,
                                c_col_idx: int, c_val: int, workspace: int, workspace_bytes: int,
                                stream: int = 0) -> None:
    _check(load().wingspan_elementwise_values(op, ctypes.byref(A), ctypes.byref(B), dtype, c_row_ptr, c_col_idx,
                                              c_val, workspace, workspace_bytes, stream or None))


def wingspan_spmspv_workspace_size(At: wingspan_csr, nnz_x: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().wingspan_spmspv_workspace_size(ctypes.byref(At), nnz_x, ctypes.byref(n)))
    return n.value


def wingspan_spmspv(At: wingspan_csr, dtype: int, x_idx: int, x_val: int, nnz_x: int, y_idx: int, y_val: int,
                    y_cap: int, workspace: int, workspace_bytes: int, stream: int = 0, check: bool = True):
    """Returns (status, y_nnz). With check=True a non-OK status raises."""
    y_nnz = ctypes.c_int64(0)
    st = load().wingspan_spmspv(ctypes.byref(At), dtype, x_idx or None, x_val or None, nnz_x, y_idx or None,
                                y_val or None, y_cap, ctypes.byref(y_nnz), workspace, workspace_bytes,
                                stream or None)
    if check:
        _check(st)
    return st, y_nnz.value


def wingspan_outer_workspace_size(At: wingspan_csr, B: wingspan_csr, products: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().wingspan_outer_workspace_size(ctypes.byref(At), ctypes.byref(B), products, ctypes.byref(n)))
    return n.value


def wingspan_outer_products(At: wingspan_csr, B: wingspan_csr, workspace: int, workspace_bytes: int,
                            stream: int = 0) -> int:
    p = ctypes.c_int64(0)
    _check(load().wingspan_outer_products(ctypes.byref(At), ctypes.byref(B), ctypes.byref(p), workspace,
                                          workspace_bytes, stream or None))
    return p.value


def wingspan_spgemm_outer(At: wingspan_csr, B: wingspan_csr, dtype: int, c_row_ptr: int, c_col_idx: int, c_val: int,
                          c_capacity: int, workspace: int, workspace_bytes: int, stream: int = 0,
                          check: bool = True):
    """Returns (status, c_nnz). With check=True a non-OK status raises."""
    nnz = ctypes.c_int64(0)
    st = load().wingspan_spgemm_outer(ctypes.byref(At), ctypes.byref(B), dtype, c_row_ptr, c_col_idx or None,
                                      c_val or None, c_capacity, ctypes.byref(nnz), workspace, workspace_bytes,
                                      stream or None)
    if check:
        _check(st)
    return st, nnz.value


# ---------------------------------------------------------------------------
# torch-level convenience: device CSR handles, allocation, both phases.
# ---------------------------------------------------------------------------

@dataclass
class DeviceCSR:
    """CSR on the GPU, held in torch tensors. Inputs use int32 row_ptr; the
    product C uses int64 row_ptr."""
    nrows: int
    ncols: int
    row_ptr: "object"
    col_idx: "object"
    val: "object"

    @property
    def nnz(self) -> int:
        return int(self.col_idx.numel())

    @property
    def dtype_code(self) -> int:
        import torch
        return F32 if self.val.dtype == torch.float32 else F64

    def desc(self) -> wingspan_csr:
        import torch
        if self.row_ptr.dtype != torch.int32:
            raise TypeError("input row_ptr must be int32")
        d = wingspan_csr()
        d.nrows, d.ncols, d.nnz = self.nrows, self.ncols, self.nnz
        d.row_ptr = self.row_ptr.data_ptr()
        d.col_idx = self.col_idx.data_ptr() if self.nnz else None
        d.val = self.val.data_ptr() if self.nnz else None
        return d

    @classmethod
    def from_host(cls, M, device="cuda") -> "DeviceCSR":
        import torch
        t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(device)
        return cls(int(M.nrows), int(M.ncols), t(M.row_ptr, np.int32), t(M.col_idx, np.int32),
                   t(M.val, M.val.dtype))

    def to_host(self):
        return HostCSR(self.nrows, self.ncols, self.row_ptr.cpu().numpy(), self.col_idx.cpu().numpy(),
                       self.val.cpu().numpy())


@dataclass
class HostCSR:
    nrows: int
    ncols: int
    row_ptr: np.ndarray
    col_idx: np.ndarray
    val: np.ndarray


def _stream_handle(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def allocate_workspace(A: DeviceCSR, B: DeviceCSR, options=None):
    import torch
    nbytes = wingspan_spgemm_workspace_size(A.desc(), B.desc(), A.dtype_code, options)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=A.row_ptr.device)
    if ws.data_ptr() % 256:
        raise RuntimeError("torch returned a workspace that is not 256-byte aligned")
    return ws, nbytes


def spgemm(A: DeviceCSR, B: DeviceCSR, options=None, stream=None, workspace=None) -> DeviceCSR:
    """C = A * B on the GPU: symbolic phase, allocate C, numeric phase."""
    import torch
    if A.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")
    dev = A.row_ptr.device
    if workspace is None:
        ws, nbytes = allocate_workspace(A, B, options)
    else:
        ws, nbytes = workspace, workspace.numel()
    h = _stream_handle(stream)
    Ad, Bd = A.desc(), B.desc()
    c_rp = torch.empty(A.nrows + 1, dtype=torch.int64, device=dev)
    nnz = wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), ws.data_ptr(), nbytes, h, options)
    c_col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(nnz, 1), dtype=A.val.dtype, device=dev)
    wingspan_spgemm_numeric(Ad, Bd, A.dtype_code, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                            ws.data_ptr(), nbytes, h, options)
    return DeviceCSR(A.nrows, B.ncols, c_rp, c_col[:nnz], c_val[:nnz])


def row_products(A: DeviceCSR, B: DeviceCSR, stream=None):
    """Per-row product counts of C = A * B on the GPU (int64 device tensor)."""
    import torch
    dev = A.row_ptr.device
    ws, nbytes = allocate_workspace(A, B)
    out = torch.empty(max(A.nrows, 1), dtype=torch.int64, device=dev)
    wingspan_spgemm_row_products(A.desc(), B.desc(), out.data_ptr(), ws.data_ptr(), nbytes, _stream_handle(stream))
    return out[:A.nrows]


@dataclass
class ShardedCSR:
    """C in sharded form: row i is pool_col[row_off[i]:row_off[i]+row_nnz[i]]
    (values at the same positions of pool_val); rows in no particular order."""
    nrows: int
    ncols: int
    row_off: "object"
    row_nnz: "object"
    pool_col: "object"
    pool_val: "object"
    nnz: int


def spgemm_sharded(A: DeviceCSR, B: DeviceCSR, options=None, stream=None, workspace=None,
                   pool_capacity: Optional[int] = None) -> ShardedCSR:
    """C = A * B in one pass with sharded output. Without pool_capacity the
    pool starts at nnz(A)+nnz(B)+64 entries and is regrown to the exact size if
    that is too small (the call is then run again)."""
    import torch
    if A.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")
    dev = A.row_ptr.device
    if workspace is None:
        ws, nbytes = allocate_workspace(A, B, options)
    else:
        ws, nbytes = workspace, workspace.numel()
    h = _stream_handle(stream)
    Ad, Bd = A.desc(), B.desc()
    row_off = torch.empty(max(A.nrows, 1), dtype=torch.int64, device=dev)
    row_nnz = torch.empty(max(A.nrows, 1), dtype=torch.int32, device=dev)
    cap = pool_capacity if pool_capacity is not None else A.nnz + B.nnz + 64
    for _ in range(2):
        pool_col = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
        pool_val = torch.empty(max(cap, 1), dtype=A.val.dtype, device=dev)
        st, used = wingspan_spgemm_sharded(Ad, Bd, A.dtype_code, row_off.data_ptr(), row_nnz.data_ptr(),
                                           pool_col.data_ptr(), pool_val.data_ptr(), cap, ws.data_ptr(), nbytes,
                                           h, options, check=False)
        if st == STATUS_CODE["WINGSPAN_ERR_INSUFFICIENT_CAPACITY"] and pool_capacity is None:
            cap = used
            continue
        _check(st)
        return ShardedCSR(A.nrows, B.ncols, row_off[:A.nrows], row_nnz[:A.nrows], pool_col, pool_val, used)
    raise RuntimeError("pool sizing did not converge")


def sharded_to_csr(S: ShardedCSR, stream=None) -> DeviceCSR:
    """Gather a sharded C into plain CSR (int64 row_ptr)."""
    import torch
    dev = S.row_off.device
    h = _stream_handle(stream)
    nbytes = wingspan_sharded_to_csr_workspace_size(S.nrows)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    c_rp = torch.empty(S.nrows + 1, dtype=torch.int64, device=dev)
    c_col = torch.empty(max(S.nnz, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(S.nnz, 1), dtype=S.pool_val.dtype, device=dev)
    dt = F32 if S.pool_val.dtype == torch.float32 else F64
    wingspan_sharded_to_csr(S.nrows, S.nnz, S.row_off.data_ptr(), S.row_nnz.data_ptr(), S.pool_col.data_ptr(),
                            S.pool_val.data_ptr(), dt, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                            ws.data_ptr(), nbytes, h)
    return DeviceCSR(S.nrows, S.ncols, c_rp, c_col[:S.nnz], c_val[:S.nnz])


def elementwise(op: str, A: DeviceCSR, B: DeviceCSR, stream=None) -> DeviceCSR:
    """C = A + B (op "add") or C = A .* B (op "hadamard") on the GPU."""
    import torch
    if A.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")
    code = {"add": OP_ADD, "hadamard": OP_HADAMARD}[op]
    dev = A.row_ptr.device
    Ad, Bd = A.desc(), B.desc()
    nbytes = wingspan_elementwise_workspace_size(Ad, Bd)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    h = _stream_handle(stream)
    c_rp = torch.empty(A.nrows + 1, dtype=torch.int64, device=dev)
    nnz = wingspan_elementwise_structure(code, Ad, Bd, c_rp.data_ptr(), ws.data_ptr(), nbytes, h)
    c_col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(nnz, 1), dtype=A.val.dtype, device=dev)
    wingspan_elementwise_values(code, Ad, Bd, A.dtype_code, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                                ws.data_ptr(), nbytes, h)
    return DeviceCSR(A.nrows, A.ncols, c_rp, c_col[:nnz], c_val[:nnz])


def spmspv(At: "DeviceCSR", x_idx, x_val, stream=None):
    """y = A x on the GPU for A given by its columns (At, the CSR of A's
    transpose) and x by device tensors of sorted int32 indices and values.
    Returns (y_idx, y_val) device tensors."""
    import torch
    if x_val.dtype != At.val.dtype:
        raise TypeError("x and A must share a value dtype")
    dev = At.row_ptr.device
    Atd = At.desc()
    nx = int(x_idx.numel())
    nbytes = wingspan_spmspv_workspace_size(Atd, nx)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    m = At.ncols
    y_idx = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    y_val = torch.empty(max(m, 1), dtype=At.val.dtype, device=dev)
    _, n = wingspan_spmspv(Atd, At.dtype_code, x_idx.data_ptr() if nx else 0, x_val.data_ptr() if nx else 0, nx,
                           y_idx.data_ptr(), y_val.data_ptr(), m, ws.data_ptr(), nbytes, _stream_handle(stream))
    return y_idx[:n], y_val[:n]


def spgemm_outer(At: "DeviceCSR", B: "DeviceCSR", stream=None) -> "DeviceCSR":
    """C = A B by outer products on the GPU, A given by its columns (At, the
    CSR of A's transpose). Counts the products, sizes the workspace, then
    computes C with the exact capacity."""
    import torch
    if At.val.dtype != B.val.dtype:
        raise TypeError("A and B must share a value dtype")
    dev = At.row_ptr.device
    Atd, Bd = At.desc(), B.desc()
    h = _stream_handle(stream)
    n0 = wingspan_outer_workspace_size(Atd, Bd, 0)
    ws0 = torch.empty(max(n0, 256), dtype=torch.uint8, device=dev)
    P = wingspan_outer_products(Atd, Bd, ws0.data_ptr(), n0, h)
    nbytes = wingspan_outer_workspace_size(Atd, Bd, P)
    del ws0
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    m = At.ncols
    c_rp = torch.empty(m + 1, dtype=torch.int64, device=dev)
    cap = P   # nnz(C) <= P
    c_col = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(cap, 1), dtype=At.val.dtype, device=dev)
    _, nnz = wingspan_spgemm_outer(Atd, Bd, At.dtype_code, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(), cap,
                                   ws.data_ptr(), nbytes, h)
    return DeviceCSR(m, B.ncols, c_rp, c_col[:nnz], c_val[:nnz])
