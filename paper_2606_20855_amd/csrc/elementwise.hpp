// Elementwise operations on two CSR matrices of one shape (paper, Section 5.2:
// SpAdd, C = A + B, and the Hadamard product, C = A .* B): a row of C is the
// sorted merge of the same rows of A and B, the union of their columns for
// the sum (an entry stored on both sides takes a + b, including an exact
// zero) and the intersection for the product.
//
// The merge is done per entry, flat over the entries: a thread takes one
// entry of A (or B), finds its row, and finds its column among the same row
// of the other matrix by binary search. That rank gives the entry's place in
// the merged row directly (the entries of the other row before it), and
// equality tells whether both sides store the column. Workgroups take chunks
// of kEwChunk consecutive entries, so long and short rows balance by
// themselves and every load and store of the entry arrays is coalesced.
#pragma once

#include "device_common.hpp"

namespace wsp {

constexpr int kEwChunk = 1024;   // entries per workgroup
constexpr int kEwRows = 1024;    // rows a chunk stages in LDS
constexpr int kEwBlock = 256;
enum EwOp { kEwAdd = 0, kEwMul = 1 };

// Last row r in [0, nrows) with rp[r] <= e (the row holding entry e when
// e < rp[nrows]). All 64 lanes of one wave take part.
__device__ __forceinline__ int wave_find_row32(const int32_t *__restrict__ rp, int nrows, int64_t e) {
    int lo = 0, hi = nrows - 1;   // rp[lo] <= e holds throughout
    while (hi > lo) {
        const int step = (hi - lo + kWave) / kWave;
        const int idx = lo + lane_id() * step;
        const bool le = idx <= hi && rp[idx] <= e;
        const uint64_t m = ballot(le);
        lo = lo + (63 - __clzll(m)) * step;   // lane 0 always qualifies
        const int h = lo + step - 1;
        hi = h < hi ? h : hi;
    }
    return lo;
}

// The rows of a chunk of entries [e0, e1): staged row pointers when there are
// at most kEwRows of them, else searched in the global row pointer.
struct ChunkRows {
    const int32_t *rp;
    const int32_t *s_rp;   // rp[r0 .. r0 + nr] when staged
    int r0, nr;
    bool staged;
    __device__ __forceinline__ int row_of(int64_t e) const {
        int lo = 0, hi = nr - 1;
        if (staged) {
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_rp[mid] <= e) lo = mid;
                else hi = mid - 1;
            }
        } else {
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (rp[r0 + mid] <= e) lo = mid;
                else hi = mid - 1;
            }
        }
        return r0 + lo;
    }
};

// All threads of the workgroup call it (it has barriers). nrows >= 1 and
// e0 < e1 <= rp[nrows].
__device__ __forceinline__ ChunkRows load_chunk_rows(const int32_t *__restrict__ rp, int nrows, int64_t e0,
                                                     int64_t e1, int32_t *s_rp, int *s_r) {
    if (threadIdx.x < kWave) {
        const int r0 = wave_find_row32(rp, nrows, e0);
        const int r1 = wave_find_row32(rp, nrows, e1 - 1);
        if (threadIdx.x == 0) {
            s_r[0] = r0;
            s_r[1] = r1;
        }
    }
    __syncthreads();
    ChunkRows cr;
    cr.rp = rp;
    cr.s_rp = s_rp;
    cr.r0 = s_r[0];
    cr.nr = s_r[1] - s_r[0] + 1;
    cr.staged = cr.nr <= kEwRows;
    if (cr.staged) {
        for (int i = threadIdx.x; i <= cr.nr; i += blockDim.x) s_rp[i] = rp[cr.r0 + i];
    }
    __syncthreads();
    return cr;
}

// First position p in [lo, hi) with col[p] >= key (hi if none).
__device__ __forceinline__ int lower_bound32(const int32_t *__restrict__ col, int lo, int hi, int key) {
    while (lo < hi) {
        const int mid = lo + ((hi - lo) >> 1);
        if (col[mid] < key) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// When dups is not null, the per-row count of the entries of A that B also
// stores (dups zeroed by the caller); when rank is not null, each A entry's
// rank in B's row, with the sign bit set when B stores the same column.
__global__ void __launch_bounds__(kEwBlock) ew_match(const int32_t *__restrict__ a_rp,
                                                     const int32_t *__restrict__ a_col,
                                                     const int32_t *__restrict__ b_rp,
                                                     const int32_t *__restrict__ b_col, int nrows, int64_t nnz_a,
                                                     int32_t *__restrict__ dups, int32_t *__restrict__ rank) {
    __shared__ int32_t s_rp[kEwRows + 1];
    __shared__ int32_t s_cnt[kEwRows];
    __shared__ int s_r[2];
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEwChunk;
    if (e0 >= nnz_a) return;   // whole workgroup
    const int64_t e1 = nnz_a - e0 < kEwChunk ? nnz_a : e0 + kEwChunk;
    for (int i = threadIdx.x; i < kEwRows; i += blockDim.x) s_cnt[i] = 0;
    const ChunkRows cr = load_chunk_rows(a_rp, nrows, e0, e1, s_rp, s_r);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
        const int r = cr.row_of(e);
        const int c = a_col[e];
        const int blo = b_rp[r], bhi = b_rp[r + 1];
        const int p = lower_bound32(b_col, blo, bhi, c);
        const bool dup = p < bhi && b_col[p] == c;
        if (rank) rank[e] = (p - blo) | (dup ? static_cast<int32_t>(0x80000000u) : 0);
        if (dup && dups) {
            if (cr.staged) atomicAdd(&s_cnt[r - cr.r0], 1);
            else atomicAdd(&dups[r], 1);
        }
    }
    __syncthreads();
    if (dups && cr.staged) {
        for (int i = threadIdx.x; i < cr.nr; i += blockDim.x)
            if (s_cnt[i]) atomicAdd(&dups[cr.r0 + i], s_cnt[i]);
    }
}

// Entries of C's rows: |A_r| + |B_r| - dups_r (sum) or dups_r (product).
struct EwCountIn {
    const int32_t *a_rp, *b_rp, *dups;
    int op;
    __device__ __forceinline__ int64_t operator()(int64_t i) const {
        const int64_t d = dups[i];
        return op == kEwAdd ? static_cast<int64_t>(a_rp[i + 1] - a_rp[i]) + (b_rp[i + 1] - b_rp[i]) - d : d;
    }
};

// 1 for an A entry that B also stores (from ew_match's rank).
struct EwDupIn {
    const int32_t *rank;
    __device__ __forceinline__ int64_t operator()(int64_t i) const { return rank[i] < 0 ? 1 : 0; }
};

// Sum. The place of an entry in its merged row is its index in its own row,
// plus the entries of the other row before its column, minus the columns both
// rows store before it (counted once). dscan is the exclusive prefix count, over
// A's entries, of those A also finds in B (ew_match's sign bit), so the common
// columns of row r before A's position q number dscan[q] - dscan[A.rp[r]].
// A's entries (rank from ew_match) write a, or a + b for a common column.
// Values are formed in double and rounded once.
template <typename V>
__global__ void __launch_bounds__(kEwBlock) ew_add_a(const int32_t *__restrict__ a_rp,
                                                     const int32_t *__restrict__ a_col,
                                                     const V *__restrict__ a_val,
                                                     const int32_t *__restrict__ b_rp,
                                                     const V *__restrict__ b_val, int nrows, int64_t nnz_a,
                                                     const int32_t *__restrict__ rank,
                                                     const int64_t *__restrict__ dscan,
                                                     const int64_t *__restrict__ c_rp, int32_t *__restrict__ c_col,
                                                     V *__restrict__ c_val) {
    __shared__ int32_t s_rp[kEwRows + 1];
    __shared__ int s_r[2];
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEwChunk;
    if (e0 >= nnz_a) return;
    const int64_t e1 = nnz_a - e0 < kEwChunk ? nnz_a : e0 + kEwChunk;
    const ChunkRows cr = load_chunk_rows(a_rp, nrows, e0, e1, s_rp, s_r);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
        const int r = cr.row_of(e);
        const int32_t k = rank[e];
        const int rb = k & 0x7fffffff;   // entries of B's row before this column
        const int ar = a_rp[r];
        const int64_t pos = c_rp[r] + (e - ar) + rb - (dscan[e] - dscan[ar]);
        double v = to_d(a_val[e]);
        if (k < 0) v += to_d(b_val[b_rp[r] + rb]);
        c_col[pos] = a_col[e];
        c_val[pos] = static_cast<V>(v);
    }
}

// Sum, B's entries: those A does not store write b (the common ones are A's).
template <typename V>
__global__ void __launch_bounds__(kEwBlock) ew_add_b(const int32_t *__restrict__ a_rp,
                                                     const int32_t *__restrict__ a_col,
                                                     const int32_t *__restrict__ b_rp,
                                                     const int32_t *__restrict__ b_col,
                                                     const V *__restrict__ b_val, int nrows, int64_t nnz_b,
                                                     const int64_t *__restrict__ dscan,
                                                     const int64_t *__restrict__ c_rp, int32_t *__restrict__ c_col,
                                                     V *__restrict__ c_val) {
    __shared__ int32_t s_rp[kEwRows + 1];
    __shared__ int s_r[2];
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEwChunk;
    if (e0 >= nnz_b) return;
    const int64_t e1 = nnz_b - e0 < kEwChunk ? nnz_b : e0 + kEwChunk;
    const ChunkRows cr = load_chunk_rows(b_rp, nrows, e0, e1, s_rp, s_r);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
        const int r = cr.row_of(e);
        const int c = b_col[e];
        const int alo = a_rp[r], ahi = a_rp[r + 1];
        const int q = lower_bound32(a_col, alo, ahi, c);   // A's entries of the row before this column end at q
        if (q < ahi && a_col[q] == c) continue;
        const int64_t pos = c_rp[r] + (e - b_rp[r]) + (q - alo) - (dscan[q] - dscan[alo]);
        c_col[pos] = c;
        c_val[pos] = b_val[e];
    }
}

// Product: an A entry that B also stores goes to pos[e] (the exclusive prefix
// count of such entries over A, which C's row-major order makes its place).
template <typename V>
__global__ void __launch_bounds__(kEwBlock) ew_mul_write(const int32_t *__restrict__ a_rp,
                                                         const int32_t *__restrict__ a_col,
                                                         const V *__restrict__ a_val,
                                                         const int32_t *__restrict__ b_rp,
                                                         const V *__restrict__ b_val, int nrows, int64_t nnz_a,
                                                         const int32_t *__restrict__ rank,
                                                         const int64_t *__restrict__ pos, int32_t *__restrict__ c_col,
                                                         V *__restrict__ c_val) {
    __shared__ int32_t s_rp[kEwRows + 1];
    __shared__ int s_r[2];
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kEwChunk;
    if (e0 >= nnz_a) return;
    const int64_t e1 = nnz_a - e0 < kEwChunk ? nnz_a : e0 + kEwChunk;
    const ChunkRows cr = load_chunk_rows(a_rp, nrows, e0, e1, s_rp, s_r);
    for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
        const int32_t k = rank[e];
        if (k >= 0) continue;
        const int r = cr.row_of(e);
        const int p = b_rp[r] + (k & 0x7fffffff);
        const int64_t q = pos[e];
        c_col[q] = a_col[e];
        c_val[q] = static_cast<V>(to_d(a_val[e]) * to_d(b_val[p]));
    }
}

}  // namespace wsp
