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

// Bucketed scatter: the products are sorted by the range of kSvRange = 4096
// positions of y their row falls in (a range is an emission tile), so each
// range can be summed in LDS by workgroups of its own, with no global atomics
// where one workgroup holds a whole range.
//   sv_bin:   a workgroup forms kSvBin products (as sv_scatter does), sorts them
//             by range in LDS (counting sort) and writes them back to its chunk
//             of tmp; tab[r * nc + c] receives chunk c's count of range r;
//   (scan):   the exclusive scan of tab in range-major order gives every
//             (range, chunk) run its place in the range-sorted order, gpos;
//   sv_place: each chunk copies its runs to their places (coalesced runs);
//   (scan):   each range is cut into pieces of at most kSvPieceMax products;
//   sv_accumulate: a workgroup takes a piece, sums it in an LDS accumulator
//             over the range's positions, and writes the sums: with plain
//             stores for a range of one piece, with global double atomics for
//             the rows it touched of a range of several, setting the flags.
constexpr int kSvRangeShift = 12;
constexpr int kSvRange = 1 << kSvRangeShift;
constexpr int kSvBin = 4096;
constexpr int kSvBinBlock = 256;
constexpr int kSvBinPer = kSvBin / kSvBinBlock;
constexpr int kSvBinStage = 2048;     // x entries a binning chunk stages in LDS
constexpr int kSvMaxRanges = 2048;    // y of at most 8 M positions takes the bucketed scatter
constexpr int kSvPieceMax = 16384;   // sorted products per accumulating workgroup at most
constexpr int kSvAccBlock = 256;
constexpr int kSvAccPer = 16;                       // products per thread and pass

// Product q's row of y and value, for a chunk whose x entries [t0, t0 + nt)
// are staged (s_pref, s_base, s_x) when nt <= kSvBinStage, else looked up in
// global memory.
template <typename V>
__device__ __forceinline__ void sv_product(const int32_t *__restrict__ at_rp, const int32_t *__restrict__ at_row,
                                           const V *__restrict__ at_val, const int32_t *__restrict__ x_idx,
                                           const V *__restrict__ x_val, const int64_t *__restrict__ pref,
                                           const int64_t *s_pref, const int64_t *s_base, const double *s_x, int t0,
                                           int nt, bool staged, int64_t q, int *row, double *v) {
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
    *row = at_row[pos];
    *v = to_d(at_val[pos]) * xv;
}

template <typename V>
__global__ void __launch_bounds__(kSvBinBlock) sv_bin(const int32_t *__restrict__ at_rp,
                                                      const int32_t *__restrict__ at_row,
                                                      const V *__restrict__ at_val,
                                                      const int32_t *__restrict__ x_idx,
                                                      const V *__restrict__ x_val, int nnz_x,
                                                      const int64_t *__restrict__ pref, const int32_t *err,
                                                      int nranges, int64_t nc, int32_t *__restrict__ tab,
                                                      int32_t *__restrict__ tmp_row, double *__restrict__ tmp_val) {
    __shared__ int32_t s_cnt[kSvMaxRanges + 1];
    __shared__ int32_t s_own[kSvBin];   // each product's x entry (relative to the chunk's first)
    // x entries staged while the products are formed, then the chunk's products sorted by range
    __shared__ __align__(16) char s_mem[kSvBin * (sizeof(int32_t) + sizeof(double))];
    __shared__ int s_t[2];
    __shared__ int32_t scratch[kSvBinBlock / kWave];
    double *s_x = reinterpret_cast<double *>(s_mem);                          // kSvBinStage entries
    int32_t *s_base = reinterpret_cast<int32_t *>(s_x + kSvBinStage);         // at_rp[x_idx[t]] - pref[t]
    int32_t *s_row = reinterpret_cast<int32_t *>(s_mem);
    double *s_val = reinterpret_cast<double *>(s_mem + kSvBin * sizeof(int32_t));
    if (*err != 0) return;   // whole grid
    const int64_t P = pref[nnz_x];
    // chunks taken grid-stride: the grid is sized for the most products x could select
    for (int64_t c = blockIdx.x; c * kSvBin < P; c += gridDim.x) {
    const int64_t q0 = c * kSvBin;
    const int64_t q1 = P - q0 < kSvBin ? P : q0 + kSvBin;
    const int n = static_cast<int>(q1 - q0);
    if (threadIdx.x < kWave) {
        const int t0 = wave_find_entry(pref, nnz_x, q0);
        const int t1 = wave_find_entry(pref, nnz_x, q1 - 1);
        if (threadIdx.x == 0) {
            s_t[0] = t0;
            s_t[1] = t1;
        }
    }
    for (int r = threadIdx.x; r < nranges; r += kSvBinBlock) s_cnt[r] = 0;
    for (int e = threadIdx.x; e < kSvBin; e += kSvBinBlock) s_own[e] = -1;
    __syncthreads();
    const int t0 = s_t[0];
    const int nt = s_t[1] - t0 + 1;
    const bool staged = nt <= kSvBinStage;
    // each x entry of the chunk with products marks the first of them in the chunk (the chunk's first
    // product belongs to entry t0), staging its column start and value when the entries fit
    for (int k0 = 0; k0 < nt; k0 += kSvBinBlock * 4) {
        int64_t pa[4], pb[4];
        int xi[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int k = k0 + static_cast<int>(threadIdx.x) + u * kSvBinBlock;
            const int t = t0 + (k < nt ? k : 0);
            pa[u] = pref[t];
            pb[u] = pref[t + 1];
            xi[u] = x_idx[t];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int k = k0 + static_cast<int>(threadIdx.x) + u * kSvBinBlock;
            if (k < nt) {
                if (pb[u] > pa[u] && pa[u] >= q0) s_own[pa[u] - q0] = k;
                if (staged) {
                    s_base[k] = static_cast<int32_t>(at_rp[xi[u]] - pa[u]);
                    s_x[k] = to_d(x_val[t0 + k]);
                }
            }
        }
    }
    __syncthreads();
    // the owners by an exclusive max-scan over the chunk's products, kSvBinPer consecutive ones per thread
    {
        const int e0 = static_cast<int>(threadIdx.x) * kSvBinPer;
        int mk[kSvBinPer];
        int x = -1;
#pragma unroll
        for (int u = 0; u < kSvBinPer; ++u) {
            mk[u] = e0 + u == 0 ? 0 : s_own[e0 + u];
            x = x > mk[u] ? x : mk[u];
        }
        int incl = wave_incl_max(x);
        const int w = threadIdx.x / kWave;
        if (lane_id() == kWave - 1) scratch[w] = incl;
        __syncthreads();
        int before = -1;
#pragma unroll
        for (int i = 0; i < kSvBinBlock / kWave; ++i) before = i < w && scratch[i] > before ? scratch[i] : before;
        int prev = __shfl_up(incl, 1, kWave);
        int run = lane_id() == 0 ? before : (prev > before ? prev : before);
#pragma unroll
        for (int u = 0; u < kSvBinPer; ++u) {
            run = run > mk[u] ? run : mk[u];
            s_own[e0 + u] = run;
        }
    }
    __syncthreads();
    int row[kSvBinPer], slot[kSvBinPer];
    double v[kSvBinPer];
    {
        // every product's A entry loaded before the first is used
        int64_t pos[kSvBinPer];
        double xv[kSvBinPer];
        if (staged) {
#pragma unroll
            for (int u = 0; u < kSvBinPer; ++u) {
                const int e = threadIdx.x + u * kSvBinBlock;
                const int k = s_own[e < n ? e : 0];
                pos[u] = static_cast<int64_t>(s_base[k]) + q0 + (e < n ? e : 0);
                xv[u] = s_x[k];
            }
        } else {
            int jx[kSvBinPer];
            int64_t pk[kSvBinPer];
#pragma unroll
            for (int u = 0; u < kSvBinPer; ++u) {
                const int e = threadIdx.x + u * kSvBinBlock;
                const int t = t0 + s_own[e < n ? e : 0];
                jx[u] = x_idx[t];
                pk[u] = pref[t];
                xv[u] = to_d(x_val[t]);
            }
#pragma unroll
            for (int u = 0; u < kSvBinPer; ++u) {
                const int e = threadIdx.x + u * kSvBinBlock;
                pos[u] = static_cast<int64_t>(at_rp[jx[u]]) + (q0 + (e < n ? e : 0) - pk[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < kSvBinPer; ++u) {
            row[u] = at_row[pos[u]];
            v[u] = to_d(at_val[pos[u]]) * xv[u];
        }
#pragma unroll
        for (int u = 0; u < kSvBinPer; ++u) {
            const int e = threadIdx.x + u * kSvBinBlock;
            if (e >= n) row[u] = -1;
            slot[u] = row[u] >= 0 ? atomicAdd(&s_cnt[row[u] >> kSvRangeShift], 1) : 0;
        }
    }
    __syncthreads();   // every count is in, and the x staging is read no more
    // the counts to the table, then their exclusive scan in place (contiguous shares per thread)
    const int per = (nranges + kSvBinBlock - 1) / kSvBinBlock;
    const int r0 = static_cast<int>(threadIdx.x) * per;
    int part = 0;
    for (int i = 0; i < per; ++i) {
        const int r = r0 + i;
        if (r < nranges) {
            const int cnt = s_cnt[r];
            tab[static_cast<int64_t>(r) * nc + c] = cnt;
            part += cnt;
        }
    }
    int total;
    int run = block_excl_scan<kSvBinBlock>(part, &total, scratch);
    for (int i = 0; i < per; ++i) {
        const int r = r0 + i;
        if (r < nranges) {
            const int cnt = s_cnt[r];
            s_cnt[r] = run;
            run += cnt;
        }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kSvBinPer; ++u) {
        if (row[u] >= 0) {
            const int k = s_cnt[row[u] >> kSvRangeShift] + slot[u];
            s_row[k] = row[u];
            s_val[k] = v[u];
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < n; e += kSvBinBlock) {
        tmp_row[q0 + e] = s_row[e];
        tmp_val[q0 + e] = s_val[e];
    }
    __syncthreads();   // LDS is reused by the next chunk
    }
}

// tab read in range-major order for the scan; chunks past the product count
// (the grid is sized by At's entries) count nothing.
struct SvTabIn {
    const int32_t *tab;
    const int64_t *pref;
    int nnz_x;
    int64_t nc;
    __device__ __forceinline__ int64_t operator()(int64_t i) const {
        const int64_t c = i % nc;
        return c * kSvBin < pref[nnz_x] ? tab[i] : 0;
    }
};

// Chunk c's runs to their places in the range-sorted order: entry e of the
// chunk (range r = its row's range) goes to gpos[r nc + c] + e - (the chunk's
// entries before range r).
__global__ void __launch_bounds__(kSvBinBlock) sv_place(const int32_t *__restrict__ tmp_row,
                                                        const double *__restrict__ tmp_val,
                                                        const int64_t *__restrict__ pref, int nnz_x,
                                                        const int32_t *err, int nranges, int64_t nc,
                                                        const int32_t *__restrict__ tab,
                                                        const int64_t *__restrict__ gpos,
                                                        int32_t *__restrict__ s_row_out,
                                                        double *__restrict__ s_val_out) {
    __shared__ int64_t s_dst[kSvMaxRanges];   // gpos of each range's run minus its first entry in the chunk
    __shared__ int32_t scratch[kSvBinBlock / kWave];
    if (*err != 0) return;
    const int64_t P = pref[nnz_x];
    for (int64_t c = blockIdx.x; c * kSvBin < P; c += gridDim.x) {
    const int64_t q0 = c * kSvBin;
    const int n = static_cast<int>(P - q0 < kSvBin ? P - q0 : kSvBin);
    const int per = (nranges + kSvBinBlock - 1) / kSvBinBlock;
    const int r0 = static_cast<int>(threadIdx.x) * per;
    int part = 0;
    for (int i = 0; i < per; ++i)
        if (r0 + i < nranges) part += tab[static_cast<int64_t>(r0 + i) * nc + c];
    int total;
    int run = block_excl_scan<kSvBinBlock>(part, &total, scratch);
    for (int i = 0; i < per; ++i) {
        const int r = r0 + i;
        if (r < nranges) {
            const int64_t k = static_cast<int64_t>(r) * nc + c;
            s_dst[r] = gpos[k] - run;
            run += tab[k];
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < n; e += kSvBinBlock) {
        const int row = tmp_row[q0 + e];
        const int64_t d = s_dst[row >> kSvRangeShift] + e;
        s_row_out[d] = row;
        s_val_out[d] = tmp_val[q0 + e];
    }
    __syncthreads();   // s_dst is reused by the next chunk
    }
}

// Range r's first place in the sorted order (r = nranges: the product count).
struct SvRangeStart {
    const int64_t *gpos;
    int64_t nc;
    __device__ __forceinline__ int64_t operator()(int r) const { return gpos[static_cast<int64_t>(r) * nc]; }
};

// The pieces of range r: its sorted products cut into runs of kSvPieceMax.
struct SvPiecesIn {
    const int64_t *gpos;
    int64_t nc;
    __device__ __forceinline__ int64_t operator()(int64_t r) const {
        const int64_t len = gpos[(r + 1) * nc] - gpos[r * nc];
        return (len + kSvPieceMax - 1) / kSvPieceMax;
    }
};

// Piece g (of piece_pre[nranges], grid-stride): range r's products
// [start + k kSvPieceMax, ...) summed in LDS, then written: with plain stores
// when the range is one piece, else its touched rows added with global double
// atomics; the flags set. yval and the flags start at zero.
__global__ void __launch_bounds__(kSvAccBlock) sv_accumulate(const int32_t *__restrict__ s_row_in,
                                                             const double *__restrict__ s_val_in,
                                                             const int32_t *err, int nranges, int64_t nc,
                                                             const int64_t *__restrict__ gpos,
                                                             const int64_t *__restrict__ piece_pre,
                                                             uint8_t *__restrict__ flag, double *__restrict__ yval) {
    __shared__ double acc[kSvRange];
    __shared__ uint8_t touched[kSvRange];
    __shared__ int s_r;
    if (*err != 0) return;
    const int64_t npieces = piece_pre[nranges];
    for (int t = threadIdx.x; t < kSvRange; t += kSvAccBlock) {
        acc[t] = 0.0;
        touched[t] = 0;
    }
    const SvRangeStart rs{gpos, nc};
    for (int64_t g = blockIdx.x; g < npieces; g += gridDim.x) {
        if (threadIdx.x < kWave) {
            // the range holding piece g (a range without pieces starts where the next one does)
            const int r = wave_last_le([=](int k) { return piece_pre[k]; }, 0, nranges - 1, g);
            if (threadIdx.x == 0) s_r = r;
        }
        __syncthreads();
        const int r = s_r;
        const int64_t b0 = rs(r), b1 = rs(r + 1);
        const int64_t k = g - piece_pre[r];
        const int64_t lo = b0 + k * kSvPieceMax;
        const int64_t hi = b1 - lo < kSvPieceMax ? b1 : lo + kSvPieceMax;
        const bool owner = piece_pre[r + 1] - piece_pre[r] == 1;
        for (int64_t k0 = lo; k0 < hi; k0 += kSvAccBlock * kSvAccPer) {
            // kSvAccPer products per thread loaded before the first is added
            int rw[kSvAccPer];
            double vl[kSvAccPer];
#pragma unroll
            for (int u = 0; u < kSvAccPer; ++u) {
                const int64_t q = k0 + threadIdx.x + u * kSvAccBlock;
                rw[u] = q < hi ? s_row_in[q] : -1;
                vl[u] = q < hi ? s_val_in[q] : 0.0;
            }
#pragma unroll
            for (int u = 0; u < kSvAccPer; ++u) {
                if (rw[u] >= 0) {
                    const int t = rw[u] & (kSvRange - 1);
                    atomicAdd(&acc[t], vl[u]);
                    touched[t] = 1;
                }
            }
        }
        __syncthreads();
        const int64_t y0 = static_cast<int64_t>(r) << kSvRangeShift;
        for (int t = threadIdx.x; t < kSvRange; t += kSvAccBlock) {
            if (touched[t]) {
                if (owner) yval[y0 + t] = acc[t];
                else unsafeAtomicAdd(&yval[y0 + t], acc[t]);
                flag[y0 + t] = 1;
                acc[t] = 0.0;
                touched[t] = 0;
            }
        }
        __syncthreads();   // the accumulator is clear for the next piece, s_r rewritable
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
