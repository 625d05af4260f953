/*
 * Test infrastructure only -- the CPU oracle for the sparse-times-sparse
 * product C = A * B (both inputs and the result in compressed rows), the
 * SpGEMM of Section 5.1 of the WingSpan paper.
 *
 * Nothing in the GPU library includes, links or calls this file. Only the
 * tests, the smoke check and the benchmark's CPU-baseline leg load it. It is
 * deliberately plain, single-threaded and slow.
 *
 * Algorithm: Gustavson's algorithm as written in the paper's SpGEMM program
 * figure (Section 5.1, Gustavson's algorithm): for every output fiber,
 * clear a dense workspace w (a SparseByteMap: dense values plus a record of
 * which positions were touched), then for each k in the input fiber and each
 * entry of the matching fiber of the other operand do w[j] += a * b, then
 * copy the touched entries of w into the output fiber in coordinate order.
 * The paper iterates column fibers of CSC matrices (j outer, then k, then i);
 * this file iterates row fibers of CSR matrices (i outer, then k, then j).
 * Row-wise Gustavson on (A, B) is the paper's column-wise Gustavson on
 * (B^T, A^T): the same loop nest over the same arrays.
 *
 * Readings where the paper is silent:
 *  - the output pattern is structural: an entry exists at (i, j) whenever some
 *    product A[i,k]*B[k,j] is formed, even if the sum is exactly zero (the
 *    workspace records touched positions, not nonzero values);
 *  - output columns are strictly increasing within each row (a SparseList
 *    level stores sorted coordinates);
 *  - every product is formed in double (exact for float inputs, the rounded
 *    double product for double inputs) and accumulated in double; float
 *    outputs are rounded once at the end;
 *  - alongside each value the oracle returns M[i,j] = sum of |products|, the
 *    quantity that bounds the rounding error of any summation order.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fused multiply-add, so a
 * product is rounded before it is added).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

enum { OR_F32 = 0, OR_F64 = 1 };

enum {
    OR_OK = 0,
    OR_ERR_ARG = -1,
    OR_ERR_ROW_PTR = -2,      /* row_ptr[0] != 0, decreasing, or row_ptr[m] != nnz */
    OR_ERR_COL_RANGE = -3,    /* column outside [0, ncols) */
    OR_ERR_COL_ORDER = -4,    /* columns not strictly increasing within a row */
    OR_ERR_NOMEM = -5,
    OR_ERR_CAPACITY = -6,
};

/* Canonical-form check of a CSR matrix with int32 row pointers and columns. */
int oracle_check_csr(int64_t nrows, int64_t ncols, int64_t nnz,
                     const int32_t *row_ptr, const int32_t *col_idx)
{
    if (nrows < 0 || ncols < 0 || nnz < 0 || !row_ptr) return OR_ERR_ARG;
    if (row_ptr[0] != 0 || (int64_t)row_ptr[nrows] != nnz) return OR_ERR_ROW_PTR;
    for (int64_t i = 0; i < nrows; ++i) {
        if (row_ptr[i + 1] < row_ptr[i]) return OR_ERR_ROW_PTR;
        for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            if (col_idx[p] < 0 || (int64_t)col_idx[p] >= ncols) return OR_ERR_COL_RANGE;
            if (p > row_ptr[i] && col_idx[p] <= col_idx[p - 1]) return OR_ERR_COL_ORDER;
        }
    }
    return OR_OK;
}

/* Number of scalar products A[i,k]*B[k,j] formed in each selected row:
 * the sum over the entries (i,k) of A of the length of row k of B. */
int oracle_row_products(const int32_t *a_rp, const int32_t *a_col,
                        const int32_t *b_rp,
                        const int64_t *rows, int64_t nsel, int64_t *out)
{
    for (int64_t s = 0; s < nsel; ++s) {
        int64_t i = rows[s];
        int64_t total = 0;
        for (int32_t a = a_rp[i]; a < a_rp[i + 1]; ++a) {
            int32_t k = a_col[a];
            total += (int64_t)(b_rp[k + 1] - b_rp[k]);
        }
        out[s] = total;
    }
    return OR_OK;
}

static int cmp_i32(const void *x, const void *y)
{
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a > b) - (a < b);
}

static double load_val(const void *v, int dtype, int64_t p)
{
    return dtype == OR_F32 ? (double)((const float *)v)[p] : ((const double *)v)[p];
}

/*
 * Gustavson over the selected rows of A (rows[0..nsel-1], any order, repeats
 * allowed), producing the matching rows of C = A * B.
 *
 * out_rp has nsel+1 entries (int64). When out_col is NULL only the row counts
 * are produced (out_rp) and no values are formed. Otherwise out_col, out_val
 * (same dtype as the inputs) and out_mag (double, may be NULL) receive the
 * entries, up to `capacity` of them.
 *
 * Returns the number of output entries, or a negative error code.
 */
int64_t oracle_spgemm_rows(int64_t ncols_b,
                           const int32_t *a_rp, const int32_t *a_col, const void *a_val,
                           const int32_t *b_rp, const int32_t *b_col, const void *b_val,
                           int dtype,
                           const int64_t *rows, int64_t nsel,
                           int64_t *out_rp, int32_t *out_col, void *out_val,
                           double *out_mag, int64_t capacity)
{
    if (ncols_b < 0 || nsel < 0 || !out_rp || (dtype != OR_F32 && dtype != OR_F64))
        return OR_ERR_ARG;
    const int values = out_col != NULL;
    size_t n = (size_t)(ncols_b > 0 ? ncols_b : 1);

    /* The workspace w: dense values, dense magnitudes, a per-position mark of
     * the last row that touched it, and the list of touched positions. */
    double *acc = values ? (double *)malloc(n * sizeof(double)) : NULL;
    double *mag = values ? (double *)malloc(n * sizeof(double)) : NULL;
    int64_t *mark = (int64_t *)malloc(n * sizeof(int64_t));
    int32_t *touched = (int32_t *)malloc(n * sizeof(int32_t));
    if (!mark || !touched || (values && (!acc || !mag))) {
        free(acc); free(mag); free(mark); free(touched);
        return OR_ERR_NOMEM;
    }
    for (size_t j = 0; j < n; ++j) mark[j] = -1;

    int64_t out = 0;
    out_rp[0] = 0;
    for (int64_t s = 0; s < nsel; ++s) {
        const int64_t i = rows[s];
        int64_t ntouched = 0;
        /* for k in row i of A (ascending), for j in row k of B (ascending) */
        for (int32_t a = a_rp[i]; a < a_rp[i + 1]; ++a) {
            const int32_t k = a_col[a];
            const double av = values ? load_val(a_val, dtype, a) : 0.0;
            for (int32_t b = b_rp[k]; b < b_rp[k + 1]; ++b) {
                const int32_t j = b_col[b];
                if (mark[j] != s) {             /* first touch of w[j] in this row */
                    mark[j] = s;
                    touched[ntouched++] = j;
                    if (values) {
                        const double p = av * load_val(b_val, dtype, b);
                        acc[j] = p;
                        mag[j] = fabs(p);
                    }
                } else if (values) {
                    const double p = av * load_val(b_val, dtype, b);
                    acc[j] += p;
                    mag[j] += fabs(p);
                }
            }
        }
        /* copy w into the output row in coordinate order */
        qsort(touched, (size_t)ntouched, sizeof(int32_t), cmp_i32);
        if (values) {
            if (out + ntouched > capacity) {
                free(acc); free(mag); free(mark); free(touched);
                return OR_ERR_CAPACITY;
            }
            for (int64_t t = 0; t < ntouched; ++t) {
                const int32_t j = touched[t];
                out_col[out + t] = j;
                if (dtype == OR_F32) ((float *)out_val)[out + t] = (float)acc[j];
                else                 ((double *)out_val)[out + t] = acc[j];
                if (out_mag) out_mag[out + t] = mag[j];
            }
        }
        out += ntouched;
        out_rp[s + 1] = out;
    }
    free(acc); free(mag); free(mark); free(touched);
    return out;
}
