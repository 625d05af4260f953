/*
 * wingspan.h -- C ABI of the MI355X (gfx950) sparse-times-sparse matrix
 * multiply C = A * B with CSR inputs and a CSR output (SpGEMM).
 *
 * The operation is the one the WingSpan paper benchmarks in Section 5.1: the
 * product of two sparse matrices whose result is stored sparse as well,
 * computed row by row with Gustavson's algorithm (Section 5.1, the four
 * SpGEMM programs figure: for each output fiber, accumulate a * b into a
 * workspace, then copy the workspace into the output fiber in coordinate
 * order).
 *
 * C[i,j] = sum over stored entries A[i,k], B[k,j] of A[i,k] * B[k,j].
 * The pattern of C is structural: (i, j) is stored whenever at least one
 * product A[i,k]*B[k,j] is formed, even if the sum is exactly zero. Columns of
 * every output row are strictly increasing.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named *_dev, and the pointers inside wingspan_csr, are HIP device
 *    pointers on the current device. Other pointers are host pointers.
 *  - The caller owns all memory. The library never allocates device memory:
 *    scratch space comes from the caller's workspace, sized by
 *    wingspan_spgemm_workspace_size(). The workspace is scratch only; its
 *    contents need not survive between calls.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream).
 *  - Every function returns a wingspan_status and never aborts or prints.
 *    Argument checks run on the host before any HIP call. On failure,
 *    wingspan_last_error() returns a message (thread-local).
 *  - Inputs must be canonical CSR: row_ptr[0] = 0, non-decreasing,
 *    row_ptr[nrows] = nnz; columns in [0, ncols), strictly increasing within
 *    each row. Non-canonical input is undefined behaviour unless
 *    options->validate is set, in which case it is detected on the device and
 *    reported as WINGSPAN_ERR_INVALID_MATRIX.
 *  - A and B may alias (C = A * A). A, B and C share one value type.
 *  - Calls on different streams with different workspaces are independent.
 */
#ifndef WINGSPAN_H
#define WINGSPAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WINGSPAN_ABI_VERSION 5

typedef enum { WINGSPAN_F32 = 0, WINGSPAN_F64 = 1 } wingspan_dtype;

typedef enum {
    WINGSPAN_OK = 0,
    WINGSPAN_ERR_INVALID_ARGUMENT = 1,    /* null pointer, negative size, bad dtype/options */
    WINGSPAN_ERR_DIMENSION_MISMATCH = 2,  /* A.ncols != B.nrows */
    WINGSPAN_ERR_INDEX_OVERFLOW = 3,      /* a size does not fit the int32 index types */
    WINGSPAN_ERR_WORKSPACE_TOO_SMALL = 4, /* workspace_bytes < wingspan_spgemm_workspace_size() */
    WINGSPAN_ERR_INSUFFICIENT_CAPACITY = 5, /* nnz(C) > c_capacity (wingspan_spgemm) or
                                             > pool_capacity (wingspan_spgemm_sharded) */
    WINGSPAN_ERR_INVALID_MATRIX = 6,      /* non-canonical input detected (options->validate) */
    WINGSPAN_ERR_HIP = 7,                 /* a HIP runtime call failed; message has the HIP error */
    WINGSPAN_ERR_UNSUPPORTED = 8,         /* a row is too long for the global spill pool, or the
                                             outer product has more than 2^31 - 1 products */
    WINGSPAN_ERR_INCONSISTENT = 9         /* numeric found a row whose entry count differs from
                                             C.row_ptr (only reported when options->validate) */
} wingspan_status;

/* A CSR matrix on the device. row_ptr has nrows+1 int32 entries, col_idx and
 * val have nnz entries; val holds float or double per the call's dtype. */
typedef struct {
    int64_t nrows;
    int64_t ncols;
    int64_t nnz;
    const int32_t *row_ptr;
    const int32_t *col_idx;
    const void *val;
} wingspan_csr;

/* Optional tuning and test switches. Pass NULL for defaults, or zero-fill the
 * struct and set version = WINGSPAN_ABI_VERSION; zero fields mean "default". */
typedef struct {
    uint32_t version;       /* must be WINGSPAN_ABI_VERSION */
    int32_t validate;       /* 1: check A and B are canonical (and, in numeric, that
                               C.row_ptr matches the product) on the device */
    int32_t max_lds_slots;  /* cap on LDS hash-table slots per row (power of two,
                               64..16384); longer rows use the dense or spill tier */
    int32_t force_spill;    /* 1: every row above the register tier uses the global
                               hash spill tier */
    int32_t window_cols;    /* dense-window width in columns: 1024, 4096, 8192 or 16384 */
    int32_t tiny_max;       /* largest per-row product count handled by the
                               register-sort tier (8..64); -1 disables that tier */
    int32_t dense_min_nnz;  /* rows with at least this many output entries (numeric) or
                               products (symbolic, single pass) use the dense tier even if
                               they fit an LDS hash table; -1 disables the dense tier; 0
                               means 2048 when the structure cache applies (1024 in its
                               symbolic phase if B has at most 262144 columns) and in a
                               single pass whose B has at most 262144 columns, else only
                               rows too large for the LDS hash tables */
    int32_t timing;         /* 1: time each tier's kernels with HIP events on `stream`
                               (the call then synchronizes the stream before returning) */
    int32_t wide_offsets;   /* 1: the dense tier forms B's entry offsets in 64 bits even
                               where 32 bits hold them (the path B takes when nnz(B) times
                               the value size exceeds 2^32); a test switch, results equal */
    int32_t cache_mib;      /* workspace budget of the structure cache, in MiB: the symbolic
                               phase keeps the column bitmaps of up to that many bytes' worth
                               of dense rows (ceil(B.ncols / 2048) * 256 bytes each) and the
                               numeric phase of the same A and B reads them instead of
                               gathering B's column indices again. 0 means 4096; -1 keeps
                               none. It changes wingspan_spgemm_workspace_size, and both
                               phases must be given the same value to share the cache. */
} wingspan_options;

/* Tiers a row can be assigned to. */
enum {
    WINGSPAN_TIER_TINY = 0,   /* one wave segment per row, register bitonic sort */
    WINGSPAN_TIER_HASH = 1,   /* one workgroup per row, LDS hash table + LDS sort */
    WINGSPAN_TIER_DENSE = 2,  /* one workgroup per row, LDS bitmap (symbolic) or dense
                                 LDS column windows (numeric) */
    WINGSPAN_TIER_SPILL = 3,  /* persistent workgroups, global-memory hash + merge sort */
    WINGSPAN_NUM_TIERS = 4
};

/* What the last symbolic (phase 0), numeric (phase 1) or single-pass
 * (phase 2, wingspan_spgemm_sharded) call on this thread did. Products are the scalar multiplies A[i,k]*B[k,j]; kernel_ms is only
 * filled when options->timing was set. */
typedef struct {
    int64_t rows[WINGSPAN_NUM_TIERS];
    int64_t a_nnz[WINGSPAN_NUM_TIERS];
    int64_t products[WINGSPAN_NUM_TIERS];
    int64_t c_nnz[WINGSPAN_NUM_TIERS];   /* numeric phase only (the single pass bins before
                                            C's row counts exist: 0) */
    int32_t launches[WINGSPAN_NUM_TIERS];
    float kernel_ms[WINGSPAN_NUM_TIERS];
    float analysis_ms;                   /* product counting, binning, scans */
    int64_t total_products;
    int64_t c_nnz_total;
    int64_t structure_cache_rows;        /* numeric phase only: dense rows whose column bitmaps the
                                            symbolic phase kept in the structure cache, which this
                                            phase's dense tier read (0: cache not used) */
} wingspan_phase_stats;

/* Bytes of device workspace the calls below need for this A, B and options.
 * Depends only on the sizes, never on the data; pure host code. */
wingspan_status wingspan_spgemm_workspace_size(const wingspan_csr *A, const wingspan_csr *B,
                                               wingspan_dtype dtype,
                                               const wingspan_options *options,
                                               size_t *bytes);

/* Symbolic phase: the number of entries of every row of C, as the exclusive
 * prefix sum c_row_ptr_dev[0..A.nrows] (int64, written by the library), and
 * the total *c_nnz (host). Synchronizes `stream` twice (once to size its
 * kernel launches, once to return *c_nnz); these are its only blocking
 * points. A.val and B.val are not read. */
wingspan_status wingspan_spgemm_symbolic(const wingspan_csr *A, const wingspan_csr *B,
                                         int64_t *c_row_ptr_dev, int64_t *c_nnz,
                                         void *workspace_dev, size_t workspace_bytes,
                                         void *stream, const wingspan_options *options);

/* Numeric phase: fills c_col_idx_dev (int32) and c_val_dev (dtype) for the
 * structure c_row_ptr_dev produced by the symbolic phase for the same A and B
 * patterns, so it can be re-run when the values of A or B change. Synchronizes
 * `stream` once (to size its kernel launches); the output kernels run
 * asynchronously. Writes never leave a row's range [c_row_ptr[i], c_row_ptr[i+1]).
 *
 * Structure cache: the symbolic phase keeps the column sets (bitmaps) of its
 * densest rows in the workspace, up to 4 GiB, with a stamp naming A and B
 * (pointers and sizes), the workspace layout and a checksum of C.row_ptr. A
 * numeric call on the same workspace whose A, B, layout and c_row_ptr_dev
 * match the stamp takes those column sets instead of recomputing them (it
 * then reads B's column indices once per product instead of twice); any other
 * call recomputes them. Calls that change A's or B's pattern in place must run
 * the symbolic phase again, as C.row_ptr itself requires. */
wingspan_status wingspan_spgemm_numeric(const wingspan_csr *A, const wingspan_csr *B,
                                        wingspan_dtype dtype, const int64_t *c_row_ptr_dev,
                                        int32_t *c_col_idx_dev, void *c_val_dev,
                                        void *workspace_dev, size_t workspace_bytes,
                                        void *stream, const wingspan_options *options);

/* Both phases. If nnz(C) exceeds c_capacity, returns
 * WINGSPAN_ERR_INSUFFICIENT_CAPACITY with c_row_ptr_dev and *c_nnz valid, so
 * the caller can allocate and call wingspan_spgemm_numeric. */
wingspan_status wingspan_spgemm(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                int64_t c_capacity, int64_t *c_nnz,
                                void *workspace_dev, size_t workspace_bytes,
                                void *stream, const wingspan_options *options);

/* ------------------------------------------------------------------------
 * wingspan_spgemm without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).
 *
 * Same arguments, results and errors as wingspan_spgemm, minus the workspace:
 * the scratch comes from a static device array of
 * WINGSPAN_NOALLOC_SCRATCH_BYTES in the library itself, one per device, held
 * from the library's first use on that device until the process ends. The
 * call allocates nothing (no hipMalloc, no library allocation). The scratch
 * holds no structure cache (the numeric phase computes its dense rows'
 * column sets itself; options->cache_mib is ignored) and a spill pool sized to what the other arrays leave.
 * A product whose scratch would exceed WINGSPAN_NOALLOC_SCRATCH_BYTES returns
 * WINGSPAN_ERR_WORKSPACE_TOO_SMALL before any HIP call; wingspan_spgemm with
 * a caller-owned workspace takes it. options->timing is refused
 * (WINGSPAN_ERR_INVALID_ARGUMENT): its events would be allocated.
 *
 * All calls on one device share that device's scratch, and each call leaves
 * its contents behind: calls that overlap in time on one device (two host
 * threads, or two streams) race and their results are undefined. Serialize
 * them. The call synchronizes `stream` as wingspan_spgemm does.
 * ------------------------------------------------------------------------ */
#define WINGSPAN_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

wingspan_status wingspan_spgemm_noalloc(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                        int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                        int64_t c_capacity, int64_t *c_nnz, void *stream,
                                        const wingspan_options *options);

/* Per-row product counts: row_products_dev[i] (int64, A.nrows entries, written
 * by the library) receives the number of scalar products A[i,k] * B[k,j] that
 * Gustavson's loop forms for row i (Section 5.1, the SpGEMM programs figure:
 * one multiply per stored A[i,k] and stored B[k,j]), i.e. the sum over the
 * entries (i, k) of A of the length of row k of B. These are the counts both
 * phases bin the rows by, from the same kernels. Takes the workspace
 * wingspan_spgemm_workspace_size() gives for (A, B) with default options;
 * asynchronous on `stream`. A.val and B.val are not read. */
wingspan_status wingspan_spgemm_row_products(const wingspan_csr *A, const wingspan_csr *B,
                                             int64_t *row_products_dev, void *workspace_dev,
                                             size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Single pass with sharded output.
 *
 * The paper's SpGEMM (Section 5.1, Gustavson's algorithm in the SpGEMM
 * programs figure) writes C into a shard level (Section 4.3, modifier levels
 * for concurrency): a fiber of the output is claimed by the one thread that
 * writes it, on its first write, and kept in that thread's own storage, so
 * no pass has to estimate the output's sparsity beforehand (Section 5.2 notes
 * the pass this saves). Here the fiber is a row of C and the writer the
 * workgroup that computes it: once the row's entries are known, the row
 * claims a contiguous segment of a caller-owned pool from a shared counter
 * and is written there, sorted by column. Rows sit in the pool in no
 * particular order. The result, "sharded CSR", is
 *
 *   row i of C = columns pool_col_dev[row_off_dev[i] .. row_off_dev[i] +
 *                row_nnz_dev[i]) with values at the same positions of
 *                pool_val_dev (dtype),
 *
 * row_off_dev int64 and row_nnz_dev int32, A.nrows entries each, written by
 * the library (rows without entries: row_nnz 0, row_off 0). A row's columns
 * are strictly increasing; the entries and values are those of
 * wingspan_spgemm, to the same rounding.
 *
 * Workspace: the same as wingspan_spgemm_workspace_size() gives for (A, B,
 * dtype, options). The pool holds pool_capacity entries (4 bytes of column
 * plus one value each). The call synchronizes `stream` twice: once to size
 * its kernel launches, once to return *pool_used.
 *
 * *pool_used (host) receives nnz(C), the entries the rows claimed. If it
 * exceeds pool_capacity the call returns WINGSPAN_ERR_INSUFFICIENT_CAPACITY:
 * row_nnz_dev is then valid, the rows that did not fit were not written, and
 * the caller can retry with a pool of *pool_used entries (an upper bound
 * beforehand is the sum over rows of min(products of the row, B.ncols)).
 * Nothing is ever written past pool_capacity.
 *
 * Dense rows (beyond the LDS hash tables) take the rank-indexed kernel only
 * when B.ncols <= 262144, where a row's entry count is known before its first
 * write; wider problems send them to the global spill tier.
 * ------------------------------------------------------------------------ */
wingspan_status wingspan_spgemm_sharded(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                        int64_t *row_off_dev, int32_t *row_nnz_dev, int32_t *pool_col_dev,
                                        void *pool_val_dev, int64_t pool_capacity, int64_t *pool_used,
                                        void *workspace_dev, size_t workspace_bytes, void *stream,
                                        const wingspan_options *options);

/* Bytes of device workspace wingspan_sharded_to_csr needs for nrows rows
 * (256-byte aligned). Pure host code. */
wingspan_status wingspan_sharded_to_csr_workspace_size(int64_t nrows, size_t *bytes);

/* Gathers a sharded C (as written by wingspan_spgemm_sharded, with every row
 * present in the pool) into plain CSR: c_row_ptr_dev (int64, nrows+1 entries)
 * is the exclusive prefix sum of row_nnz_dev, and row i's entries move to
 * [c_row_ptr[i], c_row_ptr[i+1]) of c_col_idx_dev and c_val_dev. nnz is the
 * entry count of C (the *pool_used of the sharded call; it sizes the launch);
 * the C arrays hold at least that many entries. Asynchronous on `stream`. */
wingspan_status wingspan_sharded_to_csr(int64_t nrows, int64_t nnz, const int64_t *row_off_dev,
                                        const int32_t *row_nnz_dev,
                                        const int32_t *pool_col_dev, const void *pool_val_dev, wingspan_dtype dtype,
                                        int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                        void *workspace_dev, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Elementwise operations on two CSR matrices of one shape (the paper's
 * sparse linear algebra evaluation, Section 5.2: SpAdd and the Hadamard
 * product).
 *
 *   WINGSPAN_OP_ADD:      C = A + B, stored on the union of A's and B's
 *                         coordinates; a coordinate stored on both sides takes
 *                         a + b and stays stored even when that is zero.
 *   WINGSPAN_OP_HADAMARD: C = A .* B, stored on the intersection, a * b.
 *
 * Values are formed in double and rounded once to dtype, so they equal the
 * exact sum or product correctly rounded (bit for bit the same on any
 * hardware). Rows of C have strictly increasing columns. C.row_ptr is int64.
 *
 * wingspan_elementwise_structure writes c_row_ptr_dev (A.nrows+1 entries) and
 * *c_nnz (host); it synchronizes `stream` once, to return *c_nnz. A.val and
 * B.val are not read. wingspan_elementwise_values then fills c_col_idx_dev
 * (int32) and c_val_dev, nnz(C) entries in C's row-major order, for the same
 * A and B patterns (so it can be re-run for new values); c_row_ptr_dev is the
 * array the structure call wrote, and the placement it describes is found
 * again from the patterns, so the array itself is not read. The call is
 * asynchronous. Both take the workspace wingspan_elementwise_workspace_size
 * gives (pure host code, a function of the sizes only: O(nrows + (nnz(A) +
 * nnz(B)) / 2048) bytes).
 *
 * The structure call leaves its tiling of A and B (tile boundaries and each
 * tile's place in C) in the workspace, and the library remembers that on the
 * host: a values call with the same operation, descriptors (dimensions, nnz
 * and pattern pointers; values may differ) and workspace then skips
 * recomputing it. Any other call of this library given memory that overlaps
 * the workspace forgets it. The caller must not write into the workspace, or
 * change the patterns in place, between the two calls.
 * ------------------------------------------------------------------------ */
typedef enum { WINGSPAN_OP_ADD = 0, WINGSPAN_OP_HADAMARD = 1 } wingspan_ew_op;

wingspan_status wingspan_elementwise_workspace_size(const wingspan_csr *A, const wingspan_csr *B, size_t *bytes);

wingspan_status wingspan_elementwise_structure(wingspan_ew_op op, const wingspan_csr *A, const wingspan_csr *B,
                                               int64_t *c_row_ptr_dev, int64_t *c_nnz, void *workspace_dev,
                                               size_t workspace_bytes, void *stream);

wingspan_status wingspan_elementwise_values(wingspan_ew_op op, const wingspan_csr *A, const wingspan_csr *B,
                                            wingspan_dtype dtype, const int64_t *c_row_ptr_dev,
                                            int32_t *c_col_idx_dev, void *c_val_dev, void *workspace_dev,
                                            size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Sparse matrix times sparse vector, y = A x (the paper's sparse linear
 * algebra evaluation, Section 5.2: SpMSpV, with a sparse x and a bytemap as
 * the output's root).
 *
 * A (m x n) is given by its columns: At is the CSR descriptor of A's
 * transpose (At->nrows = n, At->ncols = m; row j of At holds column j of A,
 * rows ascending). x has length n and is given by nnz_x strictly increasing
 * int32 indices x_idx_dev in [0, n) and their values x_val_dev, of the value
 * type dtype, which At.val shares. The call reads only the columns of A that
 * x selects.
 *
 * y (length m) is stored at i exactly when column j of A has an entry in row
 * i for some stored x_j, even where the sum is zero (the pattern is
 * structural); then y_i = sum over those j of A[i, j] * x_j, accumulated in
 * double (atomically, so the summation order varies between calls) and
 * rounded once to dtype. y_idx_dev (int32, strictly increasing) and y_val_dev
 * receive y's entries; *y_nnz (host) receives their count. If it exceeds y_cap
 * (y_cap = m always suffices) the call returns
 * WINGSPAN_ERR_INSUFFICIENT_CAPACITY with *y_nnz valid and only the first
 * y_cap entries written. x indices out of order or out of range give
 * WINGSPAN_ERR_INVALID_MATRIX, with y not written. The call synchronizes
 * `stream` once, to return *y_nnz. The workspace, of the size
 * wingspan_spmspv_workspace_size gives (pure host code), holds the bytemap.
 * ------------------------------------------------------------------------ */
wingspan_status wingspan_spmspv_workspace_size(const wingspan_csr *At, int64_t nnz_x, size_t *bytes);

wingspan_status wingspan_spmspv(const wingspan_csr *At, wingspan_dtype dtype, const int32_t *x_idx_dev,
                                const void *x_val_dev, int64_t nnz_x, int32_t *y_idx_dev, void *y_val_dev,
                                int64_t y_cap, int64_t *y_nnz, void *workspace_dev, size_t workspace_bytes,
                                void *stream);

/* ------------------------------------------------------------------------
 * Outer-product SpGEMM, C = A B as the sum over k of the rank-1 updates
 * A[:, k] B[k, :] (the paper's outer-product SpGEMM program, Section 5.1,
 * which runs k in parallel and guards C with a merge level: each worker
 * builds its own partial C and a coalesce step recombines them, Section 4.3).
 * The result equals the Gustavson path's C (same structure; values within
 * the rounding of a different summation order).
 *
 * A (m x K) is given by its columns: At is the CSR descriptor of A's
 * transpose (At->nrows = K, At->ncols = m); B (K x n) is CSR. The
 * intermediate storage grows with the product count
 * P = sum over k of nnz(A[:, k]) nnz(B[k, :]), so the workspace is sized in
 * two steps: wingspan_outer_workspace_size(At, B, 0, &bytes) gives what
 * wingspan_outer_products needs to count P (it synchronizes `stream` once and
 * returns P on the host); wingspan_outer_workspace_size(At, B, P, &bytes) then
 * gives the full size (pure host code, as is the first).
 *
 * wingspan_spgemm_outer counts P again (returning WINGSPAN_ERR_WORKSPACE_TOO_SMALL
 * if the workspace does not fit it) and writes c_row_ptr_dev (int64, m+1
 * entries), c_col_idx_dev (strictly increasing columns per row) and c_val_dev
 * (dtype, shared with At.val and B.val; products and sums in double, rounded
 * once); *c_nnz (host) receives nnz(C). If nnz(C) > c_capacity it returns
 * WINGSPAN_ERR_INSUFFICIENT_CAPACITY with c_row_ptr_dev and *c_nnz valid and
 * the columns and values not written. Rows of any length are merged: a row
 * whose partial entries exceed 4096 is sorted as runs of 4096 in LDS that are
 * then merged pairwise in the workspace. More than 2^31 - 1 products in all
 * gives WINGSPAN_ERR_UNSUPPORTED (the Gustavson path has no such bound). The
 * call synchronizes `stream` twice.
 * ------------------------------------------------------------------------ */
wingspan_status wingspan_outer_workspace_size(const wingspan_csr *At, const wingspan_csr *B, int64_t products,
                                              size_t *bytes);

wingspan_status wingspan_outer_products(const wingspan_csr *At, const wingspan_csr *B, int64_t *products,
                                        void *workspace_dev, size_t workspace_bytes, void *stream);

wingspan_status wingspan_spgemm_outer(const wingspan_csr *At, const wingspan_csr *B, wingspan_dtype dtype,
                                      int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                      int64_t c_capacity, int64_t *c_nnz, void *workspace_dev, size_t workspace_bytes,
                                      void *stream);

/* Statistics of the last call on this thread: phase 0 = symbolic, 1 = numeric,
 * 2 = single pass (wingspan_spgemm_sharded). */
wingspan_status wingspan_last_stats(int phase, wingspan_phase_stats *out);

/* Message for the last non-OK status on this thread ("" if none). */
const char *wingspan_last_error(void);

int wingspan_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WINGSPAN_H */
