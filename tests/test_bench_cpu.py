"""The benchmark's host-side helpers (no GPU): the algorithmic byte counts
the roofline figures divide by, the reading of the committed traffic summary,
and the refusal of a multi-GPU run."""
from __future__ import annotations

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_alg_bytes_per_unit():
    # per row: A.row_ptr and C.row_ptr entries (4 + 8); per A entry: column, value and a B.row_ptr pair
    # (4 + s + 8); per product: one B entry (4 + s); per output: one C entry (4 + s)
    for s in (4, 8):
        assert bench.alg_bytes(1, 0, 0, 0, s) == 12
        assert bench.alg_bytes(0, 1, 0, 0, s) == 12 + s
        assert bench.alg_bytes(0, 0, 1, 0, s) == 4 + s
        assert bench.alg_bytes(0, 0, 0, 1, s) == 4 + s
    assert bench.alg_bytes(3, 5, 7, 11, 4) == 3 * 12 + 5 * 16 + 7 * 8 + 11 * 8


def test_elementwise_and_spmspv_alg_bytes():
    # C = A + B, m = 2 rows, 3 + 4 entries in, 5 out, fp64: row pointers in (2 x 3 x 4) and out (3 x 8),
    # columns in (7 x 4), every value in (7 x 8), C out (5 x 12)
    assert bench.ew_alg_bytes(2, 3, 4, 5, 8, "add") == 24 + 24 + 28 + 56 + 60
    # the product reads only the common entries' values (2 per output)
    assert bench.ew_alg_bytes(2, 3, 4, 5, 8, "hadamard") == 24 + 24 + 28 + 80 + 60
    # y = A x: x entries (4 + s) and a column-pointer pair each, one A entry per product, y written once
    assert bench.sv_alg_bytes(2, 10, 3, 8) == 24 + 16 + 120 + 36


def test_measured_traffic_follows_the_source_hash(monkeypatch):
    text = open(bench.TRAFFIC_FILE).read()
    sha = [ln.split(":", 1)[1].strip() for ln in text.splitlines() if ln.startswith("- kernel_source_sha256")][0]
    want = int([ln.split(":", 1)[1].strip() for ln in text.splitlines()
                if ln.startswith("- traffic_bytes_per_launch")][0])
    monkeypatch.setattr(bench, "kernel_source_sha256", lambda: sha)
    assert bench.measured_traffic() == want
    # counters taken on another kernel source are not reported
    monkeypatch.setattr(bench, "kernel_source_sha256", lambda: "0" * 64)
    assert bench.measured_traffic() is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
