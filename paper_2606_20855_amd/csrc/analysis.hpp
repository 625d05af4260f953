// Row analysis: per-row product counts, tier/bin assignment, prefix scans,
// the column-window table of B, and optional input validation.
#pragma once

#include "device_common.hpp"

namespace wsp {

// ---------------------------------------------------------------------------
// Device-wide exclusive scan (int64 output) of a generated sequence, in three
// launches: tile sums, a scan of the tile sums, and the tile scans.
// ---------------------------------------------------------------------------
constexpr int kScanBlock = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanBlock * kScanItems;

// Length of the B row that multiplies A entry i: B.row_ptr[k+1] - B.row_ptr[k]
// with k = A.col_idx[i].
struct BRowLenIn {
    const int32_t *a_col;
    const int32_t *b_rp;
    __device__ __forceinline__ int64_t operator()(int64_t i) const {
        const int32_t k = a_col[i];
        return static_cast<int64_t>(b_rp[k + 1] - b_rp[k]);
    }
};

struct CountIn {
    const int32_t *cnt;
    __device__ __forceinline__ int64_t operator()(int64_t i) const { return cnt[i]; }
};

template <typename In>
__global__ void __launch_bounds__(kScanBlock) scan_tile_sums(In in, int64_t n, int64_t *partials) {
    __shared__ int64_t red[kScanBlock / kWave];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int64_t idx = base + static_cast<int64_t>(i) * kScanBlock + threadIdx.x;
        if (idx < n) s += in(idx);
    }
    s = block_sum<kScanBlock>(s, red);
    if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// One block: exclusive scan of partials[0..nb) in place; partials[nb] = total.
__global__ void __launch_bounds__(1024) scan_partials(int64_t *partials, int64_t nb) {
    __shared__ int64_t wsum[16];
    __shared__ int64_t carry_s;
    if (threadIdx.x == 0) carry_s = 0;
    __syncthreads();
    const int ln = lane_id();
    const int w = threadIdx.x / kWave;
    for (int64_t c0 = 0; c0 < nb; c0 += 1024) {
        const int64_t idx = c0 + threadIdx.x;
        const int64_t v = idx < nb ? partials[idx] : 0;
        int64_t incl = v;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int64_t y = __shfl_up(incl, o, kWave);
            if (ln >= o) incl += y;
        }
        if (ln == kWave - 1) wsum[w] = incl;
        __syncthreads();
        int64_t before = carry_s, tot = 0;
        for (int i = 0; i < 16; ++i) {
            before += (i < w) ? wsum[i] : 0;
            tot += wsum[i];
        }
        if (idx < nb) partials[idx] = before + incl - v;
        __syncthreads();
        if (threadIdx.x == 0) carry_s += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[nb] = carry_s;
}

// out[i] = exclusive prefix for i < n, out[n] = total.
template <typename In>
__global__ void __launch_bounds__(kScanBlock) scan_tiles(In in, int64_t n, const int64_t *partials,
                                                         int64_t nb, int64_t *out) {
    __shared__ int64_t wsum[kScanBlock / kWave];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int64_t idx = base + i;
        v[i] = idx < n ? in(idx) : 0;
        s += v[i];
    }
    const int ln = lane_id();
    const int w = threadIdx.x / kWave;
    int64_t incl = s;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(incl, o, kWave);
        if (ln >= o) incl += y;
    }
    if (ln == kWave - 1) wsum[w] = incl;
    __syncthreads();
    int64_t run = partials[blockIdx.x];
    for (int i = 0; i < kScanBlock / kWave; ++i) run += (i < w) ? wsum[i] : 0;
    run += incl - s;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int64_t idx = base + i;
        if (idx < n) out[idx] = run;
        run += v[i];
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = partials[nb];
}

// Products of row i of A: with pref the exclusive prefix of B-row lengths
// over A's entries, the row's entries [a_rp[i], a_rp[i+1]) select B rows whose
// lengths sum to pref[a_rp[i+1]] - pref[a_rp[i]].
__device__ __forceinline__ int64_t row_products_of(const int32_t *__restrict__ a_rp,
                                                   const int64_t *__restrict__ pref, int64_t i) {
    return pref[a_rp[i + 1]] - pref[a_rp[i]];
}

// out[i] = products of row i, for every row (the counts the binning uses).
__global__ void __launch_bounds__(256) row_products_kernel(const int32_t *__restrict__ a_rp,
                                                           const int64_t *__restrict__ pref, int64_t m,
                                                           int64_t *__restrict__ out) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < m) out[i] = row_products_of(a_rp, pref, i);
}

// The same exclusive scan in one workgroup of 1024 threads, for short
// sequences of cheap inputs (one launch instead of three): thread t sums its
// contiguous share, the workgroup scans the shares, and each thread writes its
// share's prefixes. out[n] = total.

template <typename In>
__global__ void __launch_bounds__(1024) scan_one_block(In in, int64_t n, int64_t *out) {
    __shared__ int64_t wsum[16];
    const int64_t per = (n + 1023) / 1024;
    const int64_t b = static_cast<int64_t>(threadIdx.x) * per;
    const int64_t e = b + per < n ? b + per : n;
    int64_t s = 0;
    for (int64_t i0 = b; i0 < e; i0 += 8) {   // eight loads in flight at a time
        int64_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = i0 + u < e ? in(i0 + u) : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    const int ln = lane_id();
    const int w = threadIdx.x / kWave;
    int64_t incl = s;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(incl, o, kWave);
        if (ln >= o) incl += y;
    }
    if (ln == kWave - 1) wsum[w] = incl;
    __syncthreads();
    int64_t run = 0, tot = 0;
    for (int i = 0; i < 16; ++i) {
        run += i < w ? wsum[i] : 0;
        tot += wsum[i];
    }
    run += incl - s;
    for (int64_t i0 = b; i0 < e; i0 += 8) {
        int64_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = i0 + u < e ? in(i0 + u) : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (i0 + u < e) out[i0 + u] = run;
            run += v[u];
        }
    }
    if (threadIdx.x == 0) out[n] = tot;
}

// ---------------------------------------------------------------------------
// Binning.
// ---------------------------------------------------------------------------
struct BinCfg {
    int64_t ncols;          // columns of B (and C)
    int64_t dense_min_nnz;  // numeric: rows with at least this many entries go dense
    int32_t tiny_max;       // 0 disables the register tier
    int32_t hash_log2_max;  // largest LDS hash table (log2 slots)
    int32_t force_spill;
    int32_t dense_ok;       // the dense tier can take rows of this problem
    int32_t numeric;        // 0: symbolic bins, 1: numeric bins
};

__device__ __forceinline__ int class_of(int64_t f) {
    // heavier rows get lower class ids (launched first)
    int l = 63 - __clzll(static_cast<unsigned long long>(f > 0 ? f : 1));
    int c = l - 10;
    c = c < 0 ? 0 : (c >= kNumClasses ? kNumClasses - 1 : c);
    return kNumClasses - 1 - c;
}

// f: products of the row; c: output entries (numeric only); bound: out, the
// hash-table bound when the row spills.
__device__ __forceinline__ int choose_bin(int64_t f, int64_t c, const BinCfg &cfg, int64_t *bound) {
    *bound = 0;
    if (f == 0) return kBinEmpty;
    if (cfg.numeric && c == 0) return kBinEmpty;
    if (f <= cfg.tiny_max) {
        const int s = f <= 8 ? 0 : (f <= 16 ? 1 : (f <= 32 ? 2 : 3));
        return kBinTiny0 + s;
    }
    int64_t need;   // table slots
    if (cfg.numeric) {
        need = c + (c >> 1);                       // load factor <= 2/3
    } else {
        const int64_t b = f < cfg.ncols ? f : cfg.ncols;   // distinct columns <= min(f, n)
        need = 2 * b;                               // load factor <= 1/2
    }
    int l = ceil_log2(need);
    if (l < kHashLog2Min) l = kHashLog2Min;
    // dense preference: numeric rows by their output entries; symbolic rows by their products (a row with c
    // entries has at least c products, so every row the numeric phase will prefer dense goes through the
    // symbolic bitmap kernel and leaves its column set in the structure cache)
    const bool dense_pref = cfg.dense_ok && (cfg.numeric ? c : f) >= cfg.dense_min_nnz;
    if (!cfg.force_spill && l <= cfg.hash_log2_max && !dense_pref) return kBinHash0 + (l - kHashLog2Min);
    if (!cfg.force_spill && cfg.dense_ok) return kBinDense0 + class_of(f);
    *bound = cfg.numeric ? c : (f < cfg.ncols ? f : cfg.ncols);
    return kBinSpill0 + class_of(f);
}

// Counts rows per bin and accumulates per-bin statistics. In the symbolic
// phase it also writes row_nnz = 0 for rows without products.
__global__ void __launch_bounds__(256) bin_count(const int32_t *__restrict__ a_rp,
                                                 const int64_t *__restrict__ pref,
                                                 const int64_t *__restrict__ c_rp, int64_t m,
                                                 BinCfg cfg, Control *ctrl,
                                                 int32_t *__restrict__ row_nnz) {
    __shared__ int32_t s_cnt[kMaxBins];
    __shared__ unsigned long long s_prod[kMaxBins], s_annz[kMaxBins], s_cnnz[kMaxBins];
    for (int i = threadIdx.x; i < kMaxBins; i += blockDim.x) {
        s_cnt[i] = 0;
        s_prod[i] = s_annz[i] = s_cnnz[i] = 0;
    }
    __syncthreads();
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < m) {
        const int32_t a0 = a_rp[i], a1 = a_rp[i + 1];
        const int64_t f = row_products_of(a_rp, pref, i);
        const int64_t c = cfg.numeric ? (c_rp[i + 1] - c_rp[i]) : 0;
        int64_t bound;
        const int b = choose_bin(f, c, cfg, &bound);
        atomicAdd(&s_cnt[b], 1);
        atomicAdd(&s_prod[b], static_cast<unsigned long long>(f));
        atomicAdd(&s_annz[b], static_cast<unsigned long long>(a1 - a0));
        atomicAdd(&s_cnnz[b], static_cast<unsigned long long>(c));
        if (bound > 0) atomicMax(reinterpret_cast<unsigned long long *>(&ctrl->spill_max_bound),
                                 static_cast<unsigned long long>(bound));
        if (!cfg.numeric && b == kBinEmpty) row_nnz[i] = 0;
    }
    __syncthreads();
    for (int b = threadIdx.x; b < kNumBins; b += blockDim.x) {
        if (s_cnt[b]) {
            atomicAdd(&ctrl->bin_count[b], s_cnt[b]);
            atomicAdd(reinterpret_cast<unsigned long long *>(&ctrl->stat_products[b]), s_prod[b]);
            atomicAdd(reinterpret_cast<unsigned long long *>(&ctrl->stat_annz[b]), s_annz[b]);
            atomicAdd(reinterpret_cast<unsigned long long *>(&ctrl->stat_cnnz[b]), s_cnnz[b]);
        }
    }
}

__global__ void bin_offsets(Control *ctrl, const int64_t *pref, int64_t nnz_a) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        int32_t run = 0;
        for (int b = 0; b < kMaxBins; ++b) {
            ctrl->bin_offset[b] = run;
            run += ctrl->bin_count[b];
        }
        ctrl->total_products = pref[nnz_a];
    }
}

// Writes each non-empty row's id into its bin's range of perm.
__global__ void __launch_bounds__(256) bin_scatter(const int32_t *__restrict__ a_rp,
                                                   const int64_t *__restrict__ pref,
                                                   const int64_t *__restrict__ c_rp, int64_t m,
                                                   BinCfg cfg, Control *ctrl,
                                                   int32_t *__restrict__ perm) {
    __shared__ int32_t s_cnt[kMaxBins];
    __shared__ int32_t s_base[kMaxBins];
    for (int b = threadIdx.x; b < kMaxBins; b += blockDim.x) s_cnt[b] = 0;
    __syncthreads();
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    int b = -1, r = 0;
    if (i < m) {
        const int64_t f = row_products_of(a_rp, pref, i);
        const int64_t c = cfg.numeric ? (c_rp[i + 1] - c_rp[i]) : 0;
        int64_t bound;
        b = choose_bin(f, c, cfg, &bound);
        if (b != kBinEmpty) r = atomicAdd(&s_cnt[b], 1);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kNumBins; k += blockDim.x)
        if (s_cnt[k]) s_base[k] = atomicAdd(&ctrl->bin_cursor[k], s_cnt[k]);
    __syncthreads();
    if (b > kBinEmpty) perm[ctrl->bin_offset[b] + s_base[b] + r] = static_cast<int32_t>(i);
}

// Zero-fill of the control block (a kernel, not a memset, so the sequence can
// be captured in a HIP graph).
__global__ void zero_words(int32_t *p, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

__global__ void fill_i64(int64_t *p, int64_t n, int64_t v) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void fill_i32(int32_t *p, int64_t n, int32_t v) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// Sharded rows to CSR: entry p of C (row r, c_rp[r] <= p < c_rp[r+1]) comes
// from pool position row_off[r] + p - c_rp[r]. Workgroup w writes entries
// [w*kGatherChunk, (w+1)*kGatherChunk) of C with coalesced stores: one wave
// finds the rows holding the chunk's ends by a 64-ary search of c_rp, the
// chunk's row pointers are staged in LDS, and each thread finds its entry's
// row by binary search there (in c_rp itself when the chunk spans very many,
// mostly empty, rows).
constexpr int kGatherChunk = 4096;
constexpr int kGatherRows = 1024;

// Last row r in [0, nrows) with c_rp[r] <= p (so c_rp[r] <= p < c_rp[r+1]
// for p < c_rp[nrows]). All 64 lanes of one wave take part.
__device__ __forceinline__ int64_t wave_find_row(const int64_t *__restrict__ c_rp, int64_t nrows, int64_t p) {
    int64_t lo = 0, hi = nrows - 1;   // c_rp[lo] <= p holds throughout
    while (hi > lo) {
        const int64_t step = (hi - lo + kWave) / kWave;   // ceil((hi - lo + 1) / 64)
        const int64_t idx = lo + static_cast<int64_t>(lane_id()) * step;
        const bool le = idx <= hi && c_rp[idx] <= p;
        const uint64_t m = ballot(le);
        const int k = 63 - __clzll(m);   // lane 0 always qualifies
        lo = lo + k * step;
        const int64_t h = lo + step - 1;
        hi = h < hi ? h : hi;
    }
    return lo;
}

template <typename V>
__global__ void __launch_bounds__(256) gather_rows(int64_t nrows, const int64_t *__restrict__ row_off,
                                                   const int64_t *__restrict__ c_rp,
                                                   const int32_t *__restrict__ pool_col,
                                                   const V *__restrict__ pool_val, int32_t *__restrict__ c_col,
                                                   V *__restrict__ c_val) {
    __shared__ int64_t s_rp[kGatherRows + 1];
    __shared__ int64_t s_off[kGatherRows];
    __shared__ int64_t s_r[2];
    const int64_t nnz = c_rp[nrows];
    const int64_t p0 = static_cast<int64_t>(blockIdx.x) * kGatherChunk;
    if (p0 >= nnz) return;   // whole workgroup leaves together
    const int64_t p1 = nnz - p0 < kGatherChunk ? nnz : p0 + kGatherChunk;
    if (threadIdx.x < kWave) {
        const int64_t r0 = wave_find_row(c_rp, nrows, p0);
        const int64_t r1 = wave_find_row(c_rp, nrows, p1 - 1);
        if (threadIdx.x == 0) {
            s_r[0] = r0;
            s_r[1] = r1;
        }
    }
    __syncthreads();
    const int64_t r0 = s_r[0], r1 = s_r[1];
    const int64_t nr = r1 - r0 + 1;
    if (nr <= kGatherRows) {
        for (int64_t i = threadIdx.x; i <= nr; i += blockDim.x) s_rp[i] = c_rp[r0 + i];
        for (int64_t i = threadIdx.x; i < nr; i += blockDim.x) s_off[i] = row_off[r0 + i];
        __syncthreads();
        for (int64_t p = p0 + threadIdx.x; p < p1; p += blockDim.x) {
            int lo = 0, hi = static_cast<int>(nr) - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_rp[mid] <= p) lo = mid;
                else hi = mid - 1;
            }
            const int64_t src = s_off[lo] + (p - s_rp[lo]);
            c_col[p] = pool_col[src];
            c_val[p] = pool_val[src];
        }
    } else {
        for (int64_t p = p0 + threadIdx.x; p < p1; p += blockDim.x) {
            int64_t lo = r0, hi = r1;
            while (lo < hi) {
                const int64_t mid = (lo + hi + 1) >> 1;
                if (c_rp[mid] <= p) lo = mid;
                else hi = mid - 1;
            }
            const int64_t src = row_off[lo] + (p - c_rp[lo]);
            c_col[p] = pool_col[src];
            c_val[p] = pool_val[src];
        }
    }
}

// Position-weighted checksum of C.row_ptr[0..m]: sum of rp[i] * (2i + 1)
// modulo 2^64, added into *out (which the caller zeroes).
__global__ void __launch_bounds__(256) rowptr_checksum(const int64_t *__restrict__ rp, int64_t m, uint64_t *out) {
    uint64_t acc = 0;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i <= m;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        acc += static_cast<uint64_t>(rp[i]) * static_cast<uint64_t>(2 * i + 1);
    acc = wave_sum(acc);
    if (lane_id() == 0) atomicAdd(reinterpret_cast<unsigned long long *>(out), static_cast<unsigned long long>(acc));
}

// Writes the stamp (one thread); magic 0 invalidates it.
__global__ void write_stamp(Stamp *stamp, Stamp value) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *stamp = value;
}

// Marks a stamp complete once its checksum has been added (one thread).
__global__ void seal_stamp(Stamp *stamp) {
    if (threadIdx.x == 0 && blockIdx.x == 0) stamp->magic = kStampMagic;
}

// Flags values that could produce a zero product: exact zeros, and (for
// double) magnitudes below 2^-537, whose products with each other could
// underflow to zero. float products are formed in double and cannot underflow.
template <typename V>
__global__ void __launch_bounds__(256) find_zero_values(const V *__restrict__ val, int64_t n, Control *ctrl) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    bool small = false;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const double v = static_cast<double>(val[i]);
        const double a = v < 0 ? -v : v;
        small |= sizeof(V) == 4 ? (a == 0.0) : !(a >= 0x1p-537);
    }
    if (__ballot(small) != 0ull && lane_id() == 0) atomicOr(&ctrl->has_zero_values, 1);
}

// ---------------------------------------------------------------------------
// Column-window table of B: wtab[k*(nwin+1) + w] is the first entry of row k
// with column >= w*wcols (w = nwin gives the row end). With it, the part of a
// row of B inside window w is one slice, found without searching.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) build_window_table(const int32_t *__restrict__ b_rp,
                                                          const int32_t *__restrict__ b_col,
                                                          int64_t nrows_b, int nwin, int wcols,
                                                          int32_t *__restrict__ wtab) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t stride = nwin + 1;
    if (t >= nrows_b * stride) return;
    const int64_t k = t / stride;
    const int w = static_cast<int>(t - k * stride);
    int lo = b_rp[k], hi = b_rp[k + 1];
    if (w < nwin) {
        const int64_t target = static_cast<int64_t>(w) * wcols;
        while (lo < hi) {
            const int mid = lo + ((hi - lo) >> 1);
            if (b_col[mid] < target) lo = mid + 1;
            else hi = mid;
        }
    } else {
        lo = hi;
    }
    wtab[t] = lo;
}

// ---------------------------------------------------------------------------
// Optional validation: one wave per row checks the row_ptr step and that the
// row's columns are in range and strictly increasing.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) validate_csr(const int32_t *__restrict__ rp,
                                                    const int32_t *__restrict__ col, int64_t nrows,
                                                    int64_t ncols, int64_t nnz, Control *ctrl) {
    const int64_t row = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
    const int ln = lane_id();
    if (row >= nrows) return;
    bool bad = false;
    const int32_t s = rp[row], e = rp[row + 1];
    if (row == 0 && s != 0) bad = true;
    if (row == nrows - 1 && static_cast<int64_t>(e) != nnz) bad = true;
    if (e < s || s < 0 || static_cast<int64_t>(e) > nnz) {
        bad = true;
    } else {
        for (int32_t p = s + ln; p < e; p += kWave) {
            const int32_t c = col[p];
            if (c < 0 || static_cast<int64_t>(c) >= ncols) bad = true;
            if (p > s && col[p - 1] >= c) bad = true;
        }
    }
    if (bad) atomicOr(&ctrl->error_flags, kErrInvalidMatrix);
}

}  // namespace wsp
