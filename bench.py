#!/usr/bin/env python3
"""SpGEMM benchmark on one MI355X: C = A*A for the R-MAT scale-18 workload.

A step is one pass of the whole hot path: the symbolic phase (product counts,
binning, per-tier entry counts, C.row_ptr scan) and the numeric phase
(re-binning and the per-tier accumulate-and-emit kernels) over the resident
input, writing into a preallocated C. Prints one JSON line:

  value      GFLOP/s of the whole step, 2 * products / step time
  roofline   the dominant numeric kernel against HBM bandwidth, from
             algorithmic bytes and its HIP-event time on the library's stream
  numeric_phase  algorithmic bytes of the numeric phase / its time
  cpu_baseline   the CPU oracle (single thread) on a seeded random sample of rows
  configs        every other SpGEMM workload: GFLOP/s, phase times, numeric
                 algorithmic GB/s against peak, the dominant kernel, and the CPU
                 oracle on the same workload (all rows, or a row sample)
  sharded_single_pass  the single pass with sharded output on the same workload
  forced_spill   the global-memory spill tier with every row above the
                 register tier forced to it
  elementwise    SpAdd and the Hadamard product (B = A, and B a shuffled copy)
                 on the R-MAT scale-20 matrix, against HBM bandwidth
  spmspv         y = A x on the same matrix with x 10% stored
  outer_product  outer-product SpGEMM on the 512x512-grid Laplacian, beside
                 the two-phase Gustavson path on the same inputs

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload rmat18]
       python bench.py --elementwise-only [--ew-workload rmat20] [--outer-workload laplace512]
       python bench.py --calibrate-copy BYTES
The second form only copies BYTES bytes device to device three times (the
runtime's plain copy kernel): run under rocprofv3 --pmc FETCH_SIZE or
WRITE_SIZE, it gives the factor that turns those counters into bytes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SpGEMM GFLOP/s (2×products/s) + effective HBM GB/s vs peak, 1 MI355X"
HBM_PEAK_GBPS = 8000.0
DEFAULT_CACHE_BYTES = 4096 << 20   # the library's structure-cache budget when options.cache_mib is 0
KERNEL_SOURCES = ["paper_2606_20855_amd/csrc/tiers.hpp", "paper_2606_20855_amd/csrc/device_common.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "numeric_dense_rmat18_traffic.md")
KERNEL_NAMES = {
    "tiny": "wsp::tiny_kernel (numeric)",
    "hash": "wsp::hash_kernel (numeric)",
    "dense": "wsp::dense_rank_kernel",
    "spill": "wsp::spill_kernel (numeric)",
}


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_sha256() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per launch of the dense numeric kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip().strip("-* `")] = v.strip().strip("`")
    if vals.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    try:
        return int(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def alg_bytes(rows, a_nnz, products, c_nnz, s):
    """Algorithmic bytes of the numeric work on these rows: A.row_ptr and
    C.row_ptr (4 + 8 per row), A entries (4 + s), a B.row_ptr pair per A entry
    (8), one B entry per product (4 + s), one C entry per output (4 + s)."""
    return 12 * rows + (12 + s) * a_nnz + (4 + s) * products + (4 + s) * c_nnz


def oracle_pass(A, B, rows=None):
    """One pass of the CPU oracle's Gustavson over `rows` (all by default),
    with the output sized beforehand by the bound sum(min(row products,
    B.ncols)) so the oracle runs once (no counting pass). Returns (seconds,
    products, output entries)."""
    import oracle
    prods = oracle.row_products(A, B, rows)
    cap = int(np.minimum(prods, B.ncols).sum())
    t0 = time.perf_counter()
    res = oracle.spgemm(A, B, rows=rows, with_mag=False, capacity=cap)
    return time.perf_counter() - t0, int(prods.sum()), res.nnz


def cpu_baseline(A, B, fraction: float, seed: int):
    rng = np.random.default_rng(seed)
    rows = np.sort(rng.choice(A.nrows, size=max(1, int(A.nrows * fraction)), replace=False)).astype(np.int64)
    dt, prods, nnz = oracle_pass(A, B, rows)
    return dict(
        value=round(2.0 * prods / dt / 1e9, 5),
        unit="GFLOP/s",
        cores=1,
        kind="oracle",
        sample=(f"{len(rows)} rows ({fraction:.0%}) drawn uniformly at random (seed {seed}) from the same "
                f"matrix; {prods} products, {nnz} output entries, {dt:.1f} s single-threaded, one pass of the "
                f"oracle"),
    )


def sharded_pass(ws, torch, dA, dB, nnz_c, P, steps, warmup, gather=True):
    """The single pass with sharded output on the same workload: each row of C
    claims its pool segment when it is done (no symbolic phase). Timed with
    HIP events on its stream, pool sized to nnz(C); the gather into plain CSR
    is timed beside it."""
    dev = dA.row_ptr.device
    Ad, Bd, dt = dA.desc(), dB.desc(), dA.dtype_code
    opts = ws.make_options(timing=1)
    wsb, nbytes = ws.allocate_workspace(dA, dB, opts)
    h = torch.cuda.current_stream().cuda_stream
    m = dA.nrows
    row_off = torch.empty(max(m, 1), dtype=torch.int64, device=dev)
    row_nnz = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    pool_col = torch.empty(max(nnz_c, 1), dtype=torch.int32, device=dev)
    pool_val = torch.empty(max(nnz_c, 1), dtype=dA.val.dtype, device=dev)

    def one():
        ws.wingspan_spgemm_sharded(Ad, Bd, dt, row_off.data_ptr(), row_nnz.data_ptr(), pool_col.data_ptr(),
                                   pool_val.data_ptr(), nnz_c, wsb.data_ptr(), nbytes, h, opts)
        return ws.wingspan_last_stats(2)

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms, tiers = [], {t: [] for t in ws.TIERS}
    for _ in range(steps):
        e0.record()
        st = one()
        e1.record()
        e1.synchronize()
        ms.append(e0.elapsed_time(e1))
        for t in ws.TIERS:
            tiers[t].append(st["kernel_ms"][t])
    # gather into CSR (needs a second copy of C beside the pool)
    to_csr_ms = None
    if gather:
        S = ws.ShardedCSR(m, dB.ncols, row_off[:m], row_nnz[:m], pool_col, pool_val, nnz_c)
        ws.sharded_to_csr(S)
        torch.cuda.synchronize()
        e0.record()
        C = ws.sharded_to_csr(S)
        e1.record()
        e1.synchronize()
        to_csr_ms = round(e0.elapsed_time(e1), 4)
        del C
    t = float(np.mean(ms))
    return dict(ms=round(t, 4), ms_min=round(float(np.min(ms)), 4), GFLOPs=round(2.0 * P / (t / 1e3) / 1e9, 2),
                tier_ms={k: round(float(np.mean(v)), 4) for k, v in tiers.items()},
                tier_rows={k: int(st["rows"][k]) for k in ws.TIERS},
                to_csr_ms=to_csr_ms, pool_entries=nnz_c)


def forced_spill_pass(ws, torch, dA, dB, steps, warmup):
    """The global-memory spill tier on a workload: every row above the
    register tier forced to it (options.force_spill), symbolic and numeric
    phases timed with HIP events, per-tier times from the library's events."""
    dev = dA.row_ptr.device
    Ad, Bd, dt = dA.desc(), dB.desc(), dA.dtype_code
    opts = ws.make_options(force_spill=1)
    topts = ws.make_options(force_spill=1, timing=1)
    wsb, nbytes = ws.allocate_workspace(dA, dB, opts)
    h = torch.cuda.current_stream().cuda_stream
    c_rp = torch.empty(dA.nrows + 1, dtype=torch.int64, device=dev)
    nnz = ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h, opts)
    c_col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(nnz, 1), dtype=dA.val.dtype, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    def step(o):
        ev[0].record()
        ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h, o)
        ev[1].record()
        ws.wingspan_spgemm_numeric(Ad, Bd, dt, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(), wsb.data_ptr(),
                                   nbytes, h, o)
        ev[2].record()
        ev[2].synchronize()
        return ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])

    for _ in range(warmup):
        step(opts)
    t = [step(opts) for _ in range(steps)]
    step(topts)
    num = ws.wingspan_last_stats(1)
    sym = ws.wingspan_last_stats(0)
    P = int(sym["total_products"])
    ts, tn = float(np.mean([x[0] for x in t])), float(np.mean([x[1] for x in t]))
    return dict(symbolic_ms=round(ts, 3), numeric_ms=round(tn, 3), GFLOPs=round(2.0 * P / ((ts + tn) / 1e3) / 1e9, 2),
                spill_rows=int(num["rows"]["spill"]), spill_products=int(num["products"]["spill"]),
                spill_launches=int(num["launches"]["spill"]),
                numeric_spill_kernel_ms=round(float(num["kernel_ms"]["spill"]), 3),
                symbolic_spill_kernel_ms=round(float(sym["kernel_ms"]["spill"]), 3))


def ew_alg_bytes(m, na, nb, nc, s, op):
    """Least HBM bytes of C = A op B in CSR: both row pointers and column
    arrays read once, C's row pointer (int64), columns and values written once;
    the sum reads every value, the product only those of the common entries."""
    vals = s * (na + nb) if op == "add" else 2 * s * nc
    return 2 * 4 * (m + 1) + 4 * (na + nb) + vals + 8 * (m + 1) + (4 + s) * nc


def elementwise_pass(ws, torch, A, workload, dev, steps, warmup, seed):
    """SpAdd and the Hadamard product on a workload's A, in the identity case
    (B = A) and the shuffled case (B = A with rows and columns relabelled by
    seeded permutations). Each op is timed whole (structure with its count
    read back, then values) and values alone, with HIP events on its stream."""
    import matgen
    dA = ws.DeviceCSR.from_host(A, dev)
    h = torch.cuda.current_stream().cuda_stream
    s = A.val.dtype.itemsize
    m = A.nrows
    Bs = matgen.shuffled_copy(A, seed)
    dBs = ws.DeviceCSR.from_host(Bs, dev)
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    out = {}
    for case, dB in (("identity", dA), ("shuffled", dBs)):
        Ad, Bd = dA.desc(), dB.desc()
        nbytes = ws.wingspan_elementwise_workspace_size(Ad, Bd)
        wsb = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
        c_rp = torch.empty(m + 1, dtype=torch.int64, device=dev)
        for op, code in (("add", ws.OP_ADD), ("hadamard", ws.OP_HADAMARD)):
            nc = ws.wingspan_elementwise_structure(code, Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h)
            c_col = torch.empty(max(nc, 1), dtype=torch.int32, device=dev)
            c_val = torch.empty(max(nc, 1), dtype=dA.val.dtype, device=dev)

            def run():
                e[0].record()
                ws.wingspan_elementwise_structure(code, Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h)
                e[1].record()
                ws.wingspan_elementwise_values(code, Ad, Bd, dA.dtype_code, c_rp.data_ptr(), c_col.data_ptr(),
                                               c_val.data_ptr(), wsb.data_ptr(), nbytes, h)
                e[2].record()
                e[2].synchronize()
                return e[0].elapsed_time(e[2]), e[1].elapsed_time(e[2])

            for _ in range(warmup):
                run()
            tot, val = zip(*[run() for _ in range(steps)])
            t = float(np.mean(tot))
            b = ew_alg_bytes(m, dA.nnz, dB.nnz, nc, s, op)
            out[f"{op}_{case}"] = dict(ms=round(t, 4), values_ms=round(float(np.mean(val)), 4), nnz_c=nc,
                                       alg_bytes=b, GBps=round(b / (t / 1e3) / 1e9, 1),
                                       frac=round(b / (t / 1e3) / 1e9 / HBM_PEAK_GBPS, 4))
            del c_col, c_val
    return dict(workload=f"{workload} A: m={A.nrows}, nnz={A.nnz}, {A.val.dtype}", **out)


def sv_alg_bytes(nx, P, ny, s):
    """Least HBM bytes of y = A x with A in compressed columns: x's entries,
    the column-pointer pair of each, the selected columns' entries, and y's
    entries written once."""
    return (4 + s) * nx + 8 * nx + (4 + s) * P + (4 + s) * ny


def spmspv_pass(ws, torch, A, workload, dev, steps, warmup, seed, density=0.1):
    """y = A x on a workload's A (given by its columns) for a seeded x with
    `density` of its entries stored (the paper's x is 90% sparse). The whole
    call is timed with HIP events on its stream (clearing the map, the
    product count read back, scatter, coalescing, y's count read back)."""
    import matgen
    At = matgen.transpose(A)
    dAt = ws.DeviceCSR.from_host(At, dev)
    xi, xv = matgen.sparse_vector(A.ncols, density, seed, A.val.dtype)
    x_idx = torch.from_numpy(xi).to(dev)
    x_val = torch.from_numpy(xv).to(dev)
    h = torch.cuda.current_stream().cuda_stream
    Atd = dAt.desc()
    nbytes = ws.wingspan_spmspv_workspace_size(Atd, len(xi))
    wsb = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    m = A.nrows
    y_idx = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    y_val = torch.empty(max(m, 1), dtype=dAt.val.dtype, device=dev)
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def run():
        e[0].record()
        _, n = ws.wingspan_spmspv(Atd, dAt.dtype_code, x_idx.data_ptr(), x_val.data_ptr(), len(xi), y_idx.data_ptr(),
                                  y_val.data_ptr(), m, wsb.data_ptr(), nbytes, h)
        e[1].record()
        e[1].synchronize()
        return e[0].elapsed_time(e[1]), n

    for _ in range(warmup):
        run()
    res = [run() for _ in range(max(steps, 5))]
    t = float(np.mean([r[0] for r in res]))
    ny = res[-1][1]
    colen = np.diff(At.row_ptr.astype(np.int64))
    P = int(colen[xi].sum())
    b = sv_alg_bytes(len(xi), P, ny, A.val.dtype.itemsize)
    return dict(workload=f"{workload} A: m={A.nrows}, nnz={A.nnz}, {A.val.dtype}; x {density:.0%} stored",
                nnz_x=len(xi), products=P, nnz_y=ny, ms=round(t, 4), ms_min=round(min(r[0] for r in res), 4),
                alg_bytes=b, GBps=round(b / (t / 1e3) / 1e9, 1), frac=round(b / (t / 1e3) / 1e9 / HBM_PEAK_GBPS, 4))


def outer_pass(ws, torch, workload, dev, steps, warmup):
    """Outer-product SpGEMM (per-workgroup partial Cs merged by a coalesce
    step) on a workload, beside the two-phase Gustavson path on the same
    inputs. Each call is timed whole with HIP events (the outer call counts its
    products and reads back nnz(C); Gustavson runs symbolic then numeric)."""
    import matgen
    A, B = matgen.config(workload)
    dAt = ws.DeviceCSR.from_host(matgen.transpose(A), dev)
    dA = ws.DeviceCSR.from_host(A, dev)
    dB = dA if B is A else ws.DeviceCSR.from_host(B, dev)
    Atd, Ad, Bd = dAt.desc(), dA.desc(), dB.desc()
    h = torch.cuda.current_stream().cuda_stream
    n0 = ws.wingspan_outer_workspace_size(Atd, Bd, 0)
    w0 = torch.empty(max(n0, 256), dtype=torch.uint8, device=dev)
    P = ws.wingspan_outer_products(Atd, Bd, w0.data_ptr(), n0, h)
    del w0
    nbytes = ws.wingspan_outer_workspace_size(Atd, Bd, P)
    wsb = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    m = A.nrows
    c_rp = torch.empty(m + 1, dtype=torch.int64, device=dev)
    c_col = torch.empty(max(P, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(P, 1), dtype=dA.val.dtype, device=dev)
    gw, gbytes = ws.allocate_workspace(dA, dB)
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def outer():
        _, nnz = ws.wingspan_spgemm_outer(Atd, Bd, dA.dtype_code, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                                          P, wsb.data_ptr(), nbytes, h)
        return nnz

    def gustavson():
        ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), gw.data_ptr(), gbytes, h, None)
        ws.wingspan_spgemm_numeric(Ad, Bd, dA.dtype_code, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                                   gw.data_ptr(), gbytes, h, None)

    def timed(fn):
        for _ in range(warmup):
            fn()
        ts = []
        for _ in range(max(steps, 5)):
            e[0].record()
            fn()
            e[1].record()
            e[1].synchronize()
            ts.append(e[0].elapsed_time(e[1]))
        return float(np.mean(ts)), float(np.min(ts))

    to, tomin = timed(outer)
    nnz = outer()
    tg, _ = timed(gustavson)
    return dict(workload=f"{workload}: m={m}, nnz(A)={A.nnz}, {A.val.dtype}", products=P, nnz_c=nnz,
                ms=round(to, 4), ms_min=round(tomin, 4), GFLOPs=round(2.0 * P / (to / 1e3) / 1e9, 2),
                gustavson_ms=round(tg, 4), vs_gustavson=round(tg / to, 3))


def host_description() -> dict:
    """The host the CPU baseline ran on: logical CPUs, model name, sockets."""
    desc = dict(nproc=os.cpu_count())
    model, sockets = None, set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name") and model is None:
                    model = line.split(":", 1)[1].strip()
                elif line.startswith("physical id"):
                    sockets.add(line.split(":", 1)[1].strip())
    except OSError:
        pass
    desc["cpu_model"] = model
    desc["sockets"] = len(sockets) or None
    return desc


def measure_spgemm(ws, torch, A, B, dev, steps, warmup, tier_steps=3):
    """One SpGEMM workload: `steps` timed steps (symbolic phase, then numeric
    phase into a preallocated C), HIP events around each phase on the
    library's stream, no per-tier timing inside the calls; then `tier_steps`
    more steps with the library's per-tier HIP events (options.timing) for the
    kernel breakdown and the dominant kernel's roofline. Options are the
    defaults, except that a workload whose dense rows' column bitmaps exceed
    the default structure-cache budget gets a budget (options.cache_mib) that
    holds them all. Returns the measurements (and the device arrays)."""
    dA = ws.DeviceCSR.from_host(A, dev)
    dB = dA if B is A else ws.DeviceCSR.from_host(B, dev)
    Ad, Bd = dA.desc(), dB.desc()
    dt = dA.dtype_code
    s = 4 if dt == ws.F32 else 8
    stream = torch.cuda.current_stream()
    h = stream.cuda_stream
    c_rp = torch.empty(A.nrows + 1, dtype=torch.int64, device=dev)
    base, cache_mib = None, 0
    wsb, nbytes = ws.allocate_workspace(dA, dB)
    nnz = ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h, None)
    need = ws.wingspan_last_stats(0)["rows"]["dense"] * (-(-B.ncols // 2048) * 256)
    if need > DEFAULT_CACHE_BYTES:
        cache_mib = -(-need // 2**20)
        base = ws.make_options(cache_mib=cache_mib)
        del wsb
        torch.cuda.empty_cache()
        wsb, nbytes = ws.allocate_workspace(dA, dB, base)
        nnz = ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h, base)
    timing = ws.make_options(timing=1, cache_mib=cache_mib)
    c_col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    c_val = torch.empty(max(nnz, 1), dtype=dA.val.dtype, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    def step(opts, e=ev):
        e[0].record(stream)
        ws.wingspan_spgemm_symbolic(Ad, Bd, c_rp.data_ptr(), wsb.data_ptr(), nbytes, h, opts)
        e[1].record(stream)
        ws.wingspan_spgemm_numeric(Ad, Bd, dt, c_rp.data_ptr(), c_col.data_ptr(), c_val.data_ptr(),
                                   wsb.data_ptr(), nbytes, h, opts)
        e[2].record(stream)

    for _ in range(warmup):
        step(base)
    torch.cuda.synchronize()
    # the timed steps follow each other without a host wait in between (the calls' own read-backs aside);
    # each step's phase events are read after the last one
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    t_start = time.perf_counter()
    for e in evs:
        step(base, e)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed / steps * 1e3
    sym_ms = [e[0].elapsed_time(e[1]) for e in evs]
    num_ms = [e[1].elapsed_time(e[2]) for e in evs]
    # per-tier kernel times (the library's events on its stream)
    tier_ms, ana_ms = {t: [] for t in ws.TIERS}, []
    for _ in range(tier_steps):
        step(timing)
        num = ws.wingspan_last_stats(1)
        sym = ws.wingspan_last_stats(0)
        ev[2].synchronize()
        ana_ms.append(num["analysis_ms"])
        for t in ws.TIERS:
            tier_ms[t].append(num["kernel_ms"][t])
    P = int(sym["total_products"])
    nnz_c = int(num["c_nnz_total"])
    b_num = alg_bytes(A.nrows, A.nnz, P, nnz_c, s)
    t_num = float(np.mean(num_ms))
    numeric_phase = dict(ms=round(t_num, 4), ms_min=round(float(np.min(num_ms)), 4), alg_bytes=b_num,
                         GBps=round(b_num / (t_num / 1e3) / 1e9, 1),
                         frac=round(b_num / (t_num / 1e3) / 1e9 / HBM_PEAK_GBPS, 4))
    dom = max(ws.TIERS, key=lambda t: np.mean(tier_ms[t]))
    k_ms = float(np.mean(tier_ms[dom]))
    launches = int(num["launches"][dom])
    b_dom = alg_bytes(num["rows"][dom], num["a_nnz"][dom], num["products"][dom], num["c_nnz"][dom], s)
    per_launch = b_dom / max(launches, 1)
    achieved = per_launch / (k_ms / max(launches, 1) / 1e3) / 1e9 if k_ms > 0 else 0.0
    roofline = dict(bound="hbm", kernel=KERNEL_NAMES[dom], achieved=round(achieved, 1), peak=HBM_PEAK_GBPS,
                    unit="GB/s", frac=round(achieved / HBM_PEAK_GBPS, 4),
                    alg_bytes_per_launch=int(per_launch), launches_per_step=launches,
                    avg_launch_ms=round(k_ms / max(launches, 1), 4))
    out = dict(
        m=A.nrows, n=B.ncols, nnz_a=A.nnz, nnz_b=B.nnz, products=P, nnz_c=nnz_c,
        value_dtype=str(A.val.dtype), accumulate="f64",
        ms_per_step=round(ms_per_step, 4), GFLOPs=round(2.0 * P / (ms_per_step / 1e3) / 1e9, 2),
        symbolic_ms=round(float(np.mean(sym_ms)), 4), numeric_ms=round(t_num, 4),
        numeric_phase=numeric_phase, roofline=roofline, dominant=dom,
        numeric_tier_ms={t: round(float(np.mean(tier_ms[t])), 4) for t in ws.TIERS},
        numeric_analysis_ms=round(float(np.mean(ana_ms)), 4),
        numeric_tier_rows={t: int(num["rows"][t]) for t in ws.TIERS},
        numeric_tier_products={t: int(num["products"][t]) for t in ws.TIERS},
        workspace_MiB=round(nbytes / 2**20, 1), cache_mib=cache_mib,
        structure_cache_rows=int(num["structure_cache_rows"]),
    )
    return out, (dA, dB)


def cpu_oracle_config(A, B, trials: int, fraction: float, seed: int):
    """The CPU oracle (single thread) on a workload: min of `trials` runs over
    all rows when fraction >= 1, else one run over a seeded random `fraction`
    of the rows, in row blocks whose outputs are dropped as they are made."""
    if fraction >= 1.0:
        runs = [oracle_pass(A, B) for _ in range(trials)]
        dt, prods = min(r[0] for r in runs), runs[0][1]
        sample = f"all {A.nrows} rows, min of {trials} one-pass runs"
    else:
        rng = np.random.default_rng(seed)
        rows = np.sort(rng.choice(A.nrows, size=max(1, int(A.nrows * fraction)), replace=False)).astype(np.int64)
        blocks = np.array_split(rows, max(1, len(rows) // 4096))
        runs = []
        for _ in range(trials):
            dt, prods = 0.0, 0
            for r in blocks:
                t, p, _ = oracle_pass(A, B, r)
                dt += t
                prods += p
            runs.append(dt)
        dt = min(runs)
        sample = (f"{len(rows)} rows ({fraction:.0%}, seed {seed}) in blocks of about 4096 rows, one pass each, "
                  f"min of {trials}")
    return dict(GFLOPs=round(2.0 * prods / dt / 1e9, 5), seconds=round(dt, 3), products=prods, cores=1,
                sample=sample)


# workloads whose single pass is timed beside their two-phase step (R-MAT 20: its dense rows span several
# 262144-column regions, so the single pass sends them to the spill tier)
SHARDED_CONFIGS = ("rmat20",)

CONFIG_CPU = {   # CPU oracle per workload: (trials, fraction of rows), each run about 0.1-10 s
    "er1000": (3, 1.0),
    "laplace512": (3, 1.0),
    "er_rect": (3, 0.2),
    "rmat18": (1, 0.1),
    "rmat20": (1, 0.01),
}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="rmat18")
    ap.add_argument("--cpu-fraction", type=float, default=0.3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES")
    ap.add_argument("--no-sharded", action="store_true", help="skip the single-pass (sharded output) timing")
    ap.add_argument("--no-elementwise", action="store_true", help="skip the SpAdd / Hadamard timing")
    ap.add_argument("--ew-workload", default="rmat20", help="the matrix A of the SpAdd / Hadamard timing")
    ap.add_argument("--elementwise-only", action="store_true",
                    help="time only SpAdd / Hadamard and SpMSpV and print their JSON objects")
    ap.add_argument("--no-spmspv", action="store_true", help="skip the SpMSpV timing")
    ap.add_argument("--no-outer", action="store_true", help="skip the outer-product SpGEMM timing")
    ap.add_argument("--outer-workload", default="laplace512", help="the workload of the outer-product timing")
    ap.add_argument("--no-spill", action="store_true", help="skip the forced spill-tier timing")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other SpGEMM workloads (timed beside the headline one in `configs`)")
    ap.add_argument("--config-steps", type=int, default=5, help="timed steps per other workload")
    ap.add_argument("--configs-only", default="", help="comma-separated workloads to time in `configs`")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibrate_copy > 0:
        src = torch.ones(args.calibrate_copy, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps(dict(calibrate_copy_bytes=args.calibrate_copy, copies=3)), flush=True)
        return

    import matgen
    from paper_2606_20855_amd import wingspan as ws

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    if args.elementwise_only:
        log(f"generating {args.ew_workload}")
        A2 = matgen.matrix(args.ew_workload)
        out = dict(steps=args.steps, warmup=args.warmup)
        log("timing SpAdd and the Hadamard product (identity and shuffled B)")
        out["elementwise"] = elementwise_pass(ws, torch, A2, args.ew_workload, dev, args.steps, args.warmup,
                                              seed=20262)
        if not args.no_spmspv:
            log("timing SpMSpV (x 10% stored)")
            out["spmspv"] = spmspv_pass(ws, torch, A2, args.ew_workload, dev, args.steps, args.warmup, seed=20263)
        if not args.no_outer:
            log("timing the outer-product SpGEMM")
            out["outer_product"] = outer_pass(ws, torch, args.outer_workload, dev, args.steps, args.warmup)
        print(json.dumps(out), flush=True)
        return
    cfg = matgen.CONFIGS[args.workload]
    t0 = time.time()
    A, B = matgen.config(args.workload)
    log(f"generated {args.workload}: m={A.nrows} nnz(A)={A.nnz} in {time.time() - t0:.1f}s")
    res, (dA, dB) = measure_spgemm(ws, torch, A, B, dev, args.steps, args.warmup)
    log(f"{args.workload}: nnz(C)={res['nnz_c']}, {res['ms_per_step']} ms per step, numeric phase "
        f"{res['numeric_ms']} ms, workspace {res['workspace_MiB']} MiB")
    P, nnz_c = res["products"], res["nnz_c"]
    roofline = dict(res["roofline"])
    roofline["traffic"] = measured_traffic() if res["dominant"] == "dense" else None
    out = dict(
        metric=METRIC,
        value=res["GFLOPs"],
        unit="GFLOP/s",
        n_gpus=1,
        steps=args.steps,
        warmup=args.warmup,
        ms_per_step=res["ms_per_step"],
        higher_is_better=True,
        scaling="weak",
        vs_baseline=None,
        dtype="f64",
        value_dtype="f32" if A.val.dtype == np.float32 else "f64",
        accumulate_dtype="f64",
        data="synthetic",
        config=dict(
            workload=f"{args.workload}: {cfg['desc']}",
            m=A.nrows, n=B.ncols, nnz_a=A.nnz, nnz_b=B.nnz, products=P, nnz_c=nnz_c,
            value_dtype=str(A.val.dtype), accumulate="f64",
            seed=cfg["seed"], options="defaults",
        ),
        roofline=roofline,
        numeric_phase=res["numeric_phase"],
        symbolic_ms=res["symbolic_ms"],
        numeric_ms=res["numeric_ms"],
        numeric_tier_ms=res["numeric_tier_ms"],
        numeric_analysis_ms=res["numeric_analysis_ms"],
        numeric_tier_rows=res["numeric_tier_rows"],
        numeric_tier_products=res["numeric_tier_products"],
    )
    if not args.no_sharded:
        log("timing the single pass with sharded output")
        torch.cuda.empty_cache()
        sh = sharded_pass(ws, torch, dA, dB, nnz_c, P, args.steps, args.warmup)
        sh["vs_two_phase_step"] = round(res["ms_per_step"] / sh["ms"], 3)
        sh["vs_two_phase_step_with_gather"] = round(res["ms_per_step"] / (sh["ms"] + sh["to_csr_ms"]), 3)
        out["sharded_single_pass"] = sh
    if not args.no_spill:
        log("timing the spill tier (every row above the register tier forced to it)")
        torch.cuda.empty_cache()
        out["forced_spill"] = forced_spill_pass(ws, torch, dA, dB, max(2, args.steps // 3), 1)
    del dA, dB
    torch.cuda.empty_cache()
    if not (args.no_elementwise and args.no_spmspv):
        A2 = matgen.matrix(args.ew_workload)
        if not args.no_elementwise:
            log("timing SpAdd and the Hadamard product (identity and shuffled B)")
            out["elementwise"] = elementwise_pass(ws, torch, A2, args.ew_workload, dev, args.steps, args.warmup,
                                                  seed=20262)
        if not args.no_spmspv:
            log("timing SpMSpV (x 10% stored)")
            out["spmspv"] = spmspv_pass(ws, torch, A2, args.ew_workload, dev, args.steps, args.warmup, seed=20263)
        del A2
        torch.cuda.empty_cache()
    if not args.no_outer:
        log("timing the outer-product SpGEMM")
        out["outer_product"] = outer_pass(ws, torch, args.outer_workload, dev, args.steps, args.warmup)
    host = host_description()
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a row sample")
        cb = cpu_baseline(A, B, args.cpu_fraction, seed=20261)
        cb.update(host=host)
        out["cpu_baseline"] = cb
    if not args.no_configs:
        names = [n for n in (args.configs_only.split(",") if args.configs_only else matgen.CONFIGS)
                 if n and n != args.workload]
        out["configs"] = {}
        for name in names:
            ccfg = matgen.CONFIGS[name]
            t0 = time.time()
            Ac, Bc = matgen.config(name)
            log(f"timing {name}: m={Ac.nrows} nnz(A)={Ac.nnz} (generated in {time.time() - t0:.1f}s)")
            r, (dAc, dBc) = measure_spgemm(ws, torch, Ac, Bc, dev, args.config_steps, 1)
            r["workload"] = f"{name}: {ccfg['desc']}"
            torch.cuda.empty_cache()
            if name in SHARDED_CONFIGS and not args.no_sharded:
                log(f"timing the single pass with sharded output on {name}")
                c_bytes = r["nnz_c"] * (4 + (4 if Ac.val.dtype == np.float32 else 8))
                sh = sharded_pass(ws, torch, dAc, dBc, r["nnz_c"], r["products"], 2, 1, gather=2 * c_bytes < 150e9)
                sh["vs_two_phase_step"] = round(r["ms_per_step"] / sh["ms"], 3)
                if sh["to_csr_ms"] is not None:
                    sh["vs_two_phase_step_with_gather"] = round(r["ms_per_step"] / (sh["ms"] + sh["to_csr_ms"]), 3)
                r["sharded_single_pass"] = sh
            del dAc, dBc
            torch.cuda.empty_cache()
            if not args.no_cpu_baseline:
                trials, frac = CONFIG_CPU[name]
                log(f"timing the CPU oracle on {name}")
                r["cpu_oracle"] = cpu_oracle_config(Ac, Bc, trials, frac, seed=20264)
                r["cpu_oracle"]["gpu_vs_cpu"] = round(r["GFLOPs"] / max(r["cpu_oracle"]["GFLOPs"], 1e-12), 1)
            out["configs"][name] = r
            del Ac, Bc
        if not args.no_cpu_baseline:
            out["configs_cpu_host"] = host
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
