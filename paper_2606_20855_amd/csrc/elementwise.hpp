// Elementwise operations on two CSR matrices of one shape (paper, Section 5.2:
// SpAdd, C = A + B, and the Hadamard product, C = A .* B): a row of C is the
// sorted merge of the same rows of A and B, the union of their columns for
// the sum (an entry stored on both sides takes a + b, including an exact
// zero) and the intersection for the product.
//
// A and B are read as one merged sequence: all entries of both in row-major
// (row, column) order, A's entry first where both store a coordinate. The
// sequence is cut into tiles of kEwTile entries by merge-path splits
// (ew_tile_splits: the row holding a boundary found on the summed row
// pointers, then a split of that row's two column lists), a boundary that
// would separate the two entries of a common coordinate taking the B entry
// along. A tile's shares of A and of B are contiguous runs of their entry
// arrays, so a workgroup loads both with coalesced reads into LDS as
// (row, column) keys and matches them there:
//   ew_tile_count: the coordinates both sides store, per tile (and per row,
//                  for C's row pointer);
//   ew_tile_write: each entry's place in C, from its rank among the other
//                  side's share and the common coordinates before it, after
//                  the tile's first place (a scan of the tiles' counts).
// Long and short rows balance by themselves; nothing but the entries, the
// row pointers and C is read or written at the size of the inputs.
#pragma once

#include "search.hpp"

namespace wsp {

constexpr int kEwTile = 2048;    // merged entries per tile (one more when a common coordinate straddles)
constexpr int kEwBlock = 256;
constexpr int kEwRows = 1024;    // rows whose common coordinates a tile counts in LDS (more: global atomics)
constexpr int kEwPer = (kEwTile + 1 + kEwBlock - 1) / kEwBlock;   // consecutive tile positions per thread
enum EwOp { kEwAdd = 0, kEwMul = 1 };
constexpr int64_t kEwEnd = 0x7fffffffffffffffll;   // above every (row, column) key

// Tile boundaries, one wave each: for t in [0, ntiles], d = min(t kEwTile,
// nnz(A) + nnz(B)); split_a[t] and split_b[t] count the A and B entries before
// boundary t and split_r[t] is the row holding it (nrows - 1 at the end).
// nrows >= 1.
__global__ void __launch_bounds__(256) ew_tile_splits(const int32_t *__restrict__ a_rp,
                                                      const int32_t *__restrict__ a_col,
                                                      const int32_t *__restrict__ b_rp,
                                                      const int32_t *__restrict__ b_col, int nrows, int64_t ntiles,
                                                      int64_t *__restrict__ split_a, int64_t *__restrict__ split_b,
                                                      int32_t *__restrict__ split_r) {
    const int64_t t = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    if (t > ntiles) return;   // whole wave
    const int64_t na_all = a_rp[nrows], nb_all = b_rp[nrows];
    const int64_t total = na_all + nb_all;
    const int64_t d = t * kEwTile < total ? t * kEwTile : total;
    int64_t ia = na_all, ib = nb_all;
    int r = nrows - 1;
    if (d < total) {
        r = wave_last_le([=](int k) { return static_cast<int64_t>(a_rp[k]) + b_rp[k]; }, 0, nrows - 1, d);
        const int64_t ar = a_rp[r], br = b_rp[r];
        const int64_t na = a_rp[r + 1] - ar, nb = b_rp[r + 1] - br;
        const int64_t dd = d - ar - br;   // < na + nb: row r holds position d
        const int64_t i = wave_merge_split(a_col + ar, na, b_col + br, nb, dd);
        int64_t j = dd - i;
        if (i > 0 && j < nb && a_col[ar + i - 1] == b_col[br + j]) ++j;   // keep a common pair together
        ia = ar + i;
        ib = br + j;
    }
    if (lane_id() == 0) {
        split_a[t] = ia;
        split_b[t] = ib;
        split_r[t] = r;
    }
}

// A tile's shares and rows: A entries [ia0, ia0 + na), B entries
// [ib0, ib0 + nb), all in rows [r0, r0 + nr).
struct EwTile {
    int64_t ia0, ib0;
    int na, nb, r0, nr;
};

__device__ __forceinline__ EwTile ew_tile_of(const int64_t *__restrict__ split_a, const int64_t *__restrict__ split_b,
                                             const int32_t *__restrict__ split_r) {
    const int t = blockIdx.x;
    EwTile T;
    T.ia0 = split_a[t];
    T.ib0 = split_b[t];
    T.na = static_cast<int>(split_a[t + 1] - T.ia0);
    T.nb = static_cast<int>(split_b[t + 1] - T.ib0);
    T.r0 = split_r[t];
    T.nr = split_r[t + 1] - T.r0 + 1;
    return T;
}

// A DPP lane move of an unsigned value; lanes with no source read 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, ROW_MASK, 0xf, false));
}

// Inclusive wave max-scan of unsigned values (identity 0): row shifts within
// 16-lane rows, then row broadcasts of lanes 15 and 31.
__device__ __forceinline__ uint32_t wave_incl_umax(uint32_t v) {
    v = max(v, dpp_u32<kDppRowShr1, 0xf>(v));
    v = max(v, dpp_u32<kDppRowShr2, 0xf>(v));
    v = max(v, dpp_u32<kDppRowShr4, 0xf>(v));
    v = max(v, dpp_u32<kDppRowShr8, 0xf>(v));
    v = max(v, dpp_u32<kDppRowBcast15, 0xa>(v));
    v = max(v, dpp_u32<kDppRowBcast31, 0xc>(v));
    return v;
}

// Exclusive block-wide max-scan of unsigned values (0 for thread 0).
// `scratch` holds BLOCK/64 ints.
template <int BLOCK>
__device__ __forceinline__ uint32_t block_excl_umax(uint32_t x, int *scratch) {
    constexpr int NW = BLOCK / kWave;
    const uint32_t incl = wave_incl_umax(x);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) scratch[w] = static_cast<int>(incl);
    __syncthreads();
    uint32_t before = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) before = i < w ? max(before, static_cast<uint32_t>(scratch[i])) : before;
    __syncthreads();
    const uint32_t prev = static_cast<uint32_t>(__shfl_up(static_cast<int>(incl), 1, kWave));
    return max(before, lane_id() == 0 ? 0u : prev);
}

// Loads a tile as (row, column) keys in LDS, A's share at [0, na) and B's at
// [na, na + nb) (with VALS, values in double beside them): the columns, with
// coalesced reads, into the keys' low halves, and, at the same time, the row
// pointers of the tile's rows. Then each row that starts inside a share marks
// its first position in the key's high half (row r0 + k as k + 1 in A's
// share, nr + k + 1 in B's, so one max-scan over both shares serves and B's
// marks exceed all of A's), and an exclusive max-scan over the positions,
// kEwPer consecutive ones per thread, replaces the marks by the rows. All
// threads call it.
template <bool VALS, typename V>
__device__ __forceinline__ void ew_load_tile(const EwTile &T, const int32_t *__restrict__ a_rp,
                                             const int32_t *__restrict__ a_col, const V *__restrict__ a_val,
                                             const int32_t *__restrict__ b_rp, const int32_t *__restrict__ b_col,
                                             const V *__restrict__ b_val, int64_t *s_key, double *s_val,
                                             int *scratch) {
    uint32_t *half = reinterpret_cast<uint32_t *>(s_key);   // [2p] column, [2p + 1] mark, then row
    const int n = T.na + T.nb;
    const uint32_t nr = static_cast<uint32_t>(T.nr);
    // the first kEwBlock rows' pointers, read beside the columns
    const int k0 = threadIdx.x;
    int64_t sa0 = -1, ea0 = -1, sb0 = -1, eb0 = -1;
    if (k0 < T.nr) {
        sa0 = a_rp[T.r0 + k0] - T.ia0;
        ea0 = a_rp[T.r0 + k0 + 1] - T.ia0;
        sb0 = b_rp[T.r0 + k0] - T.ib0;
        eb0 = b_rp[T.r0 + k0 + 1] - T.ib0;
    }
    // position p of the tile (A's share, then B's), kEwPer per thread strided by the block: all loads
    // issued before the first is waited for
    int32_t col[kEwPer];
    double val[kEwPer];
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        const int p = threadIdx.x + u * kEwBlock;
        col[u] = 0;
        val[u] = 0.0;
        if (p < T.na) {
            col[u] = a_col[T.ia0 + p];
            if (VALS) val[u] = to_d(a_val[T.ia0 + p]);
        } else if (p < n) {
            col[u] = b_col[T.ib0 + (p - T.na)];
            if (VALS) val[u] = to_d(b_val[T.ib0 + (p - T.na)]);
        }
    }
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        const int p = threadIdx.x + u * kEwBlock;
        if (p < n) {
            s_key[p] = static_cast<uint32_t>(col[u]);
            if (VALS) s_val[p] = val[u];
        }
    }
    __syncthreads();
    // a non-empty row starting inside a share is the only one to mark that position
    if (k0 < T.nr) {
        if (sa0 >= 0 && sa0 < T.na && ea0 > sa0) half[2 * sa0 + 1] = static_cast<uint32_t>(k0) + 1u;
        if (sb0 >= 0 && sb0 < T.nb && eb0 > sb0) half[2 * (T.na + sb0) + 1] = nr + static_cast<uint32_t>(k0) + 1u;
    }
    for (int k = k0 + blockDim.x; k < T.nr; k += blockDim.x) {   // tiles over many empty rows
        const int64_t sa = a_rp[T.r0 + k] - T.ia0, ea = a_rp[T.r0 + k + 1] - T.ia0;
        if (sa >= 0 && sa < T.na && ea > sa) half[2 * sa + 1] = static_cast<uint32_t>(k) + 1u;
        const int64_t sb = b_rp[T.r0 + k] - T.ib0, eb = b_rp[T.r0 + k + 1] - T.ib0;
        if (sb >= 0 && sb < T.nb && eb > sb) half[2 * (T.na + sb) + 1] = nr + static_cast<uint32_t>(k) + 1u;
    }
    __syncthreads();
    const int p0 = threadIdx.x * kEwPer;
    uint32_t mk[kEwPer];
    uint32_t x = 0;
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        const int p = p0 + u;
        uint32_t v = p < n ? half[2 * p + 1] : 0u;
        if (p == 0 && T.na > 0) v = max(v, 1u);             // A's share starts in row r0
        if (p == T.na && T.nb > 0) v = max(v, nr + 1u);     // and so does B's
        mk[u] = v;
        x = max(x, v);
    }
    uint32_t run = block_excl_umax<kEwBlock>(x, scratch);
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        const int p = p0 + u;
        run = max(run, mk[u]);
        if (p < n) half[2 * p + 1] = static_cast<uint32_t>(T.r0) + (p < T.na ? run - 1u : run - nr - 1u);
    }
    __syncthreads();
}

// Merge-path split inside a tile: the number of A's share among the first d
// entries of the tile's merged order (A first on equal keys).
__device__ __forceinline__ int ew_split(const int64_t *s_key, int na, int nb, int d) {
    int lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (s_key[mid] > s_key[na + d - mid - 1]) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

// Per tile: tile_cnt[t] = C's entries from the tile (the shares' sizes less
// the common coordinates for the sum, the common coordinates for the
// product). With PER_ROW, also each row's common coordinates added to
// dups[row] (zeroed by the caller).
template <bool PER_ROW>
__global__ void __launch_bounds__(kEwBlock) ew_tile_count(const int32_t *__restrict__ a_rp,
                                                          const int32_t *__restrict__ a_col,
                                                          const int32_t *__restrict__ b_rp,
                                                          const int32_t *__restrict__ b_col,
                                                          const int64_t *__restrict__ split_a,
                                                          const int64_t *__restrict__ split_b,
                                                          const int32_t *__restrict__ split_r, int op,
                                                          int32_t *__restrict__ tile_cnt, int32_t *__restrict__ dups) {
    __shared__ int64_t s_key[kEwTile + 1];
    __shared__ int32_t s_cnt[PER_ROW ? kEwRows : 1];
    __shared__ int32_t scratch[kEwBlock / kWave];
    const EwTile T = ew_tile_of(split_a, split_b, split_r);
    const bool local = PER_ROW && T.nr <= kEwRows;
    if (local)
        for (int k = threadIdx.x; k < T.nr; k += blockDim.x) s_cnt[k] = 0;
    ew_load_tile<false, float>(T, a_rp, a_col, nullptr, b_rp, b_col, nullptr, s_key, nullptr, scratch);
    const int n = T.na + T.nb;
    const int d = threadIdx.x * kEwPer;
    int c = 0;
    if (d < n) {
        int i = ew_split(s_key, T.na, T.nb, d), j = d - i;
        int64_t ka = i < T.na ? s_key[i] : kEwEnd, kb = j < T.nb ? s_key[T.na + j] : kEwEnd;
        const int steps = n - d < kEwPer ? n - d : kEwPer;
        for (int u = 0; u < steps; ++u) {
            if (ka <= kb) {
                if (ka == kb) {
                    ++c;
                    if (PER_ROW) {
                        const int row = static_cast<int>(ka >> 32);
                        if (local) atomicAdd(&s_cnt[row - T.r0], 1);
                        else atomicAdd(&dups[row], 1);
                    }
                }
                ++i;
                ka = i < T.na ? s_key[i] : kEwEnd;
            } else {
                ++j;
                kb = j < T.nb ? s_key[T.na + j] : kEwEnd;
            }
        }
    }
    c = block_sum<kEwBlock>(c, scratch);   // (its barriers also order the LDS counts)
    if (threadIdx.x == 0) tile_cnt[blockIdx.x] = op == kEwAdd ? n - c : c;
    if (local)
        for (int k = threadIdx.x; k < T.nr; k += blockDim.x)
            if (s_cnt[k]) atomicAdd(&dups[T.r0 + k], s_cnt[k]);
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

struct EwTileIn {
    const int32_t *cnt;
    __device__ __forceinline__ int64_t operator()(int64_t t) const { return cnt[t]; }
};

// C's entries from a tile, from tile_off[t] on: each thread walks kEwPer
// consecutive positions of the tile's merged order (from a merge-path split),
// keeping, for the sum, every entry but the B half of a common coordinate (the
// A half takes a + b) and, for the product, the A half of each common
// coordinate (a * b). The kept entries' values are then read (all loads of a
// thread issued together, overlapping the scan of the kept counts that places
// them), formed in double and rounded once, and the tile's part of C is
// staged in LDS and written with coalesced stores.
template <typename V, int OP>
__global__ void __launch_bounds__(kEwBlock) ew_tile_write(const int32_t *__restrict__ a_rp,
                                                          const int32_t *__restrict__ a_col,
                                                          const V *__restrict__ a_val,
                                                          const int32_t *__restrict__ b_rp,
                                                          const int32_t *__restrict__ b_col,
                                                          const V *__restrict__ b_val,
                                                          const int64_t *__restrict__ split_a,
                                                          const int64_t *__restrict__ split_b,
                                                          const int32_t *__restrict__ split_r,
                                                          const int64_t *__restrict__ tile_off,
                                                          int32_t *__restrict__ c_col, V *__restrict__ c_val) {
    __shared__ int64_t s_key[kEwTile + 1];
    __shared__ int32_t s_ocol[kEwTile + 1];
    __shared__ int32_t scratch[kEwBlock / kWave];
    const EwTile T = ew_tile_of(split_a, split_b, split_r);
    ew_load_tile<false, V>(T, a_rp, a_col, nullptr, b_rp, b_col, nullptr, s_key, nullptr, scratch);
    const int n = T.na + T.nb;
    const int d = threadIdx.x * kEwPer;
    int32_t oc[kEwPer];
    int ai[kEwPer], bi[kEwPer];   // the kept entry's A and B share indices (-1: that side stores nothing)
    int c = 0;
    int i = 0, j = 0;
    if (d < n) {
        i = ew_split(s_key, T.na, T.nb, d);
        j = d - i;
    }
    // the current A and B keys (kEwEnd past a share's end) and the last A key before j's entry
    int64_t ka = i < T.na ? s_key[i] : kEwEnd, kb = j < T.nb ? s_key[T.na + j] : kEwEnd;
    int64_t prev_a = i > 0 ? s_key[i - 1] : -1;
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        oc[u] = 0;
        ai[u] = -1;
        bi[u] = -1;
        bool keep = false;
        if (d + u < n) {
            if (ka <= kb) {
                const bool common = ka == kb;
                keep = OP == kEwAdd || common;
                oc[u] = static_cast<int32_t>(ka & 0xffffffffll);
                ai[u] = keep ? i : -1;
                bi[u] = keep && common ? j : -1;
                prev_a = ka;
                ++i;
                ka = i < T.na ? s_key[i] : kEwEnd;
            } else {
                keep = OP == kEwAdd && prev_a != kb;   // else the B half of a common coordinate
                oc[u] = static_cast<int32_t>(kb & 0xffffffffll);
                bi[u] = keep ? j : -1;
                ++j;
                kb = j < T.nb ? s_key[T.na + j] : kEwEnd;
            }
        }
        c += keep;
    }
    double av[kEwPer], bv[kEwPer];
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        av[u] = ai[u] >= 0 ? to_d(a_val[T.ia0 + ai[u]]) : 0.0;
        bv[u] = bi[u] >= 0 ? to_d(b_val[T.ib0 + bi[u]]) : 0.0;
    }
    int tot;
    int p = block_excl_scan<kEwBlock>(c, &tot, scratch);   // (its barriers end every thread's walk)
    // the tile's entries of C staged in LDS in order (values over the keys), then written coalesced
    V *s_oval = reinterpret_cast<V *>(s_key);
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        if (ai[u] >= 0 || bi[u] >= 0) {
            double v;
            if (OP == kEwMul) v = av[u] * bv[u];
            else v = ai[u] >= 0 && bi[u] >= 0 ? av[u] + bv[u] : (ai[u] >= 0 ? av[u] : bv[u]);
            s_ocol[p] = oc[u];
            s_oval[p] = static_cast<V>(v);
            ++p;
        }
    }
    __syncthreads();
    const int64_t base = tile_off[blockIdx.x];
#pragma unroll
    for (int u = 0; u < kEwPer; ++u) {
        const int e = threadIdx.x + u * kEwBlock;
        if (e < tot) {
            c_col[base + e] = s_ocol[e];
            c_val[base + e] = s_oval[e];
        }
    }
}

}  // namespace wsp
