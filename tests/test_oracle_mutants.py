"""Sensitivity of the oracle's pins: plant plausible mistakes in copies of the
oracle's C source (on the CPU only) and check that the independent checks
used by the pin tests reject every one of them."""
import os
import subprocess

import numpy as np
import pytest

import matgen
import oracle
from matgen import CSR

SRC = os.path.join(os.path.dirname(oracle.__file__), "spgemm_oracle.c")

# (name, original text, planted mistake)
MUTANTS = [
    ("dropped_term", "acc[j] += p;", "acc[j] = p;"),
    ("wrong_sign", "acc[j] += p;", "acc[j] -= p;"),
    ("first_product_dropped", "acc[j] = p;\n                        mag[j] = fabs(p);",
     "acc[j] = 0.0;\n                        mag[j] = fabs(p);"),
    ("wrong_b_index", "const double p = av * load_val(b_val, dtype, b);\n                    acc[j] += p;",
     "const double p = av * load_val(b_val, dtype, b > 0 ? b - 1 : b);\n                    acc[j] += p;"),
    ("wrong_column_index", "const int32_t j = b_col[b];", "const int32_t j = b_col[b_rp[k]];"),
    ("no_sort", "qsort(touched,", "if (0) qsort(touched,"),
    ("stale_workspace", "if (mark[j] != s) {", "if (mark[j] < 0) {"),
    ("skipped_last_b", "b < b_rp[k + 1]; ++b)", "b + 1 < b_rp[k + 1]; ++b)"),
    ("skipped_first_a", "for (int32_t a = a_rp[i]; a < a_rp[i + 1]; ++a) {\n            const int32_t k = a_col[a];\n            const double av",
     "for (int32_t a = a_rp[i] + 1; a < a_rp[i + 1]; ++a) {\n            const int32_t k = a_col[a];\n            const double av"),
    ("float_accumulator", "const double p = av * load_val(b_val, dtype, b);\n                    acc[j] += p;",
     "const double p = av * load_val(b_val, dtype, b);\n                    acc[j] = (double)(float)(acc[j] + p);"),
]


def _pins_pass(lib) -> bool:
    """The independent checks: dense brute force (values, structure, counts)
    on rectangular inputs with empty rows, in both precisions."""
    for seed, (m, k, n), dtype in [(1, (9, 13, 11), np.float64), (2, (20, 30, 25), np.float32),
                                   (3, (16, 16, 16), np.float64)]:
        A = matgen.random_sparse(m, k, 0.4, seed, dtype, "pm1", empty_rows=0.2)
        B = matgen.random_sparse(k, n, 0.4, seed + 10, dtype, "pm1", empty_rows=0.2)
        try:
            res = oracle.spgemm(A, B, lib=lib)
        except RuntimeError:
            return False
        Ad, Bd = A.to_dense(), B.to_dense()
        pat = (A.pattern_dense() @ B.pattern_dense()) > 0
        rp = res.row_ptr
        if rp[-1] != pat.sum():
            return False
        got = CSR(m, n, rp, res.col_idx, np.ones(res.nnz)).pattern_dense() > 0
        if not np.array_equal(pat, got):
            return False
        for i in range(m):
            if np.any(np.diff(res.col_idx[rp[i]:rp[i + 1]]) <= 0):
                return False
        rows = np.repeat(np.arange(m), np.diff(rp))
        ref = (Ad @ Bd)[rows, res.col_idx]
        mag = (np.abs(Ad) @ np.abs(Bd))[rows, res.col_idx]
        eps = 1e-13 if dtype == np.float64 else 1.2e-7
        if not np.all(np.abs(res.val - ref) <= eps * mag):
            return False
    return True


def test_unmutated_oracle_passes():
    assert _pins_pass(None)


@pytest.mark.parametrize("name,orig,bad", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, orig, bad):
    src = open(SRC).read()
    assert orig in src, f"mutation site for {name} not found"
    mutated = src.replace(orig, bad, 1)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(mutated)
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(so), str(c), "-lm"])
    lib = oracle._bind(str(so))
    assert not _pins_pass(lib), f"planted mistake {name} was not detected"
