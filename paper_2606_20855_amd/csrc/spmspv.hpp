// Sparse matrix times sparse vector, y = A x (paper, Section 5.2: SpMSpV with
// a merged bytemap as the output's root). A comes in compressed columns (the
// CSR arrays of its transpose, At: row j of At is column j of A), so the
// products of a stored x_j are the entries of one row of At, read with
// coalesced loads, and only the columns x selects are touched.
//
// The output is a bytemap over y's m positions (a stored flag per position
// and a double accumulator), which every thread updates: the paper guards it
// with a merge level (a copy per thread, recombined at the end); here the
// hardware's global double atomics recombine the updates as they happen, and
// the flags mark the positions written. The map is then coalesced into the
// sorted sparse y by a scan of the flags.
//
// Products are processed flat: product q belongs to the x entry t with
// pref[t] <= q < pref[t+1] (pref: exclusive prefix of the selected columns'
// lengths), so long and short columns balance by themselves.
#pragma once

#include "analysis.hpp"
#include "search.hpp"

namespace wsp {

constexpr int kSvChunk = 512;    // products per workgroup
constexpr int kSvStage = 512;    // x entries a chunk stages in LDS
constexpr int kSvBlock = 256;

// Length of the column of A that x entry t selects. It also checks x: an
// index outside [0, n), or not above the one before it, sets
// kErrInvalidMatrix in *err (and counts 0, so nothing reads past At).
struct SvLenIn {
    const int32_t *at_rp, *x_idx;
    int64_t n;
    int32_t *err;
    __device__ __forceinline__ int64_t operator()(int64_t t) const {
        const int j = x_idx[t];
        const bool bad = j < 0 || j >= n || (t > 0 && x_idx[t - 1] >= j);
        if (bad) {
            atomicOr(err, kErrInvalidMatrix);
            return 0;
        }
        return static_cast<int64_t>(at_rp[j + 1] - at_rp[j]);
    }
};

// Clears the map (flags as int32 words, accumulators) and the error word.
__global__ void __launch_bounds__(256) sv_clear(int32_t *__restrict__ flag_words, int64_t nwords,
                                                int64_t *__restrict__ yval_bits, int64_t m, int32_t *err) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < nwords) flag_words[i] = 0;
    if (i < m) yval_bits[i] = 0;
    if (i == 0) *err = 0;
}

// 1 where y is stored.
struct SvFlagIn {
    const uint8_t *flag;
    __device__ __forceinline__ int64_t operator()(int64_t i) const { return flag[i] != 0 ? 1 : 0; }
};

// Scatters the P = pref[nnz_x] products into the map: yval[i] += A[i, j] * x_j
// and flag[i] = 1 for each selected entry (i, j). Workgroups take chunks of
// kSvChunk products, grid-stride, reading P (and the check of x, which stops
// everything) from device memory, so the host need not wait for them. A
// chunk's x entries are staged in LDS when they number at most kSvStage: their
// first product, their column's start in At minus that, and x_j. Values are
// multiplied and accumulated in double.
template <typename V>
__global__ void __launch_bounds__(kSvBlock) sv_scatter(const int32_t *__restrict__ at_rp,
                                                       const int32_t *__restrict__ at_row,
                                                       const V *__restrict__ at_val,
                                                       const int32_t *__restrict__ x_idx,
                                                       const V *__restrict__ x_val, int nnz_x,
                                                       const int64_t *__restrict__ pref, const int32_t *err,
                                                       uint8_t *__restrict__ flag, double *__restrict__ yval) {
    __shared__ int64_t s_pref[kSvStage + 1];
    __shared__ int64_t s_base[kSvStage];
    __shared__ double s_x[kSvStage];
    __shared__ int s_t[2];
    if (*err != 0) return;   // whole grid
    const int64_t P = pref[nnz_x];
    for (int64_t q0 = static_cast<int64_t>(blockIdx.x) * kSvChunk; q0 < P;
         q0 += static_cast<int64_t>(gridDim.x) * kSvChunk) {
        const int64_t q1 = P - q0 < kSvChunk ? P : q0 + kSvChunk;
        if (threadIdx.x < kWave) {
            const int t0 = wave_find_entry(pref, nnz_x, q0);
            const int t1 = wave_find_entry(pref, nnz_x, q1 - 1);
            if (threadIdx.x == 0) {
                s_t[0] = t0;
                s_t[1] = t1;
            }
        }
        __syncthreads();
        const int t0 = s_t[0];
        const int nt = s_t[1] - t0 + 1;
        const bool staged = nt <= kSvStage;
        if (staged) {
            for (int k = threadIdx.x; k < nt; k += blockDim.x) {
                const int t = t0 + k;
                const int64_t p = pref[t];
                s_pref[k] = p;
                s_base[k] = static_cast<int64_t>(at_rp[x_idx[t]]) - p;
                s_x[k] = to_d(x_val[t]);
            }
        }
        __syncthreads();
        for (int64_t q = q0 + threadIdx.x; q < q1; q += blockDim.x) {
            int64_t pos;
            double xv;
            if (staged) {
                int lo = 0, hi = nt - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (s_pref[mid] <= q) lo = mid;
                    else hi = mid - 1;
                }
                pos = s_base[lo] + q;
                xv = s_x[lo];
            } else {
                int lo = t0, hi = t0 + nt - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (pref[mid] <= q) lo = mid;
                    else hi = mid - 1;
                }
                pos = static_cast<int64_t>(at_rp[x_idx[lo]]) + (q - pref[lo]);
                xv = to_d(x_val[lo]);
            }
            const int i = at_row[pos];
            unsafeAtomicAdd(&yval[i], to_d(at_val[pos]) * xv);
            flag[i] = 1;
        }
        __syncthreads();   // the chunk's staging is read no more
    }
}

// The map is coalesced into y tile by tile: kSvTile positions per workgroup.
// sv_tile_count counts a tile's stored positions (its flags read as 32-bit
// words); once the counts are scanned (tile_pre, with the total at
// tile_pre[ntiles]), sv_emit_tiles writes each tile's stored positions to
// y[tile_pre[t] + rank within the tile] when that is below cap, values rounded
// once to the value type.
constexpr int kSvTile = 4096;
constexpr int kSvTileBlock = 256;

__global__ void __launch_bounds__(kSvTileBlock) sv_tile_count(const uint32_t *__restrict__ flag_words, int64_t m,
                                                             int32_t *__restrict__ tile_cnt) {
    __shared__ int32_t red[kSvTileBlock / kWave];
    const int64_t w0 = static_cast<int64_t>(blockIdx.x) * (kSvTile / 4);
    const int64_t nw = (m + 3) / 4;
    int c = 0;
    for (int k = threadIdx.x; k < kSvTile / 4; k += kSvTileBlock) {
        const int64_t w = w0 + k;
        if (w < nw) {
            const uint32_t f = flag_words[w];   // one flag byte (0 or 1) per position
            c += static_cast<int>((f & 1u) + ((f >> 8) & 1u) + ((f >> 16) & 1u) + (f >> 24));
        }
    }
    c = block_sum<kSvTileBlock>(c, red);
    if (threadIdx.x == 0) tile_cnt[blockIdx.x] = c;
}

struct SvTileIn {
    const int32_t *cnt;
    __device__ __forceinline__ int64_t operator()(int64_t t) const { return cnt[t]; }
};

template <typename V>
__global__ void __launch_bounds__(kSvTileBlock) sv_emit_tiles(const uint8_t *__restrict__ flag,
                                                             const double *__restrict__ yval,
                                                             const int64_t *__restrict__ tile_pre, int64_t m,
                                                             int64_t cap, int32_t *__restrict__ y_idx,
                                                             V *__restrict__ y_val) {
    __shared__ int32_t scratch[kSvTileBlock / kWave];
    constexpr int PER = kSvTile / kSvTileBlock;   // consecutive positions per thread
    const int64_t i0 = static_cast<int64_t>(blockIdx.x) * kSvTile + static_cast<int64_t>(threadIdx.x) * PER;
    bool f[PER];
    int c = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int64_t i = i0 + k;
        f[k] = i < m && flag[i] != 0;
        c += f[k];
    }
    int tot;
    int64_t p = tile_pre[blockIdx.x] + block_excl_scan<kSvTileBlock>(c, &tot, scratch);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        if (f[k]) {
            if (p < cap) {
                y_idx[p] = static_cast<int32_t>(i0 + k);
                y_val[p] = static_cast<V>(yval[i0 + k]);
            }
            ++p;
        }
    }
}

}  // namespace wsp
