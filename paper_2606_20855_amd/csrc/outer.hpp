// Outer-product SpGEMM, C = A B = sum over k of A[:, k] B[k, :] (paper,
// Section 5.1: the outer-product program of the SpGEMM figure, which runs
// the contraction index k in parallel and guards C with a merge level, a copy
// of C per worker recombined by `coalesce`, Section 4.3).
//
// A comes by its columns (At, the CSR arrays of A's transpose) and B by its
// rows, so the rank-1 update of index k pairs row k of At with row k of B.
// Its |At_k| * |B_k| products, over all k, are numbered flat (q over the
// exclusive prefix pref of the per-k counts) and cut into chunks of kOpChunk:
//   1. each workgroup forms its chunk's products, sorts them by (row, column)
//      in LDS and sums equal coordinates: the workgroup's own partial C;
//   2. coalesce: every partial entry moves to its row's bucket (the partial
//      C's rows concatenated, in arbitrary order), then each row's bucket is
//      sorted by column and equal columns summed: in registers up to 64
//      entries, in LDS up to kOpRowCap, and beyond that as runs of kOpRowCap
//      sorted in LDS then merged pairwise in global memory (merge path, each
//      output tile merged in LDS);
//   3. the compacted rows are scanned into C.row_ptr and gathered into CSR.
// Products are formed and summed in double; values are rounded once.
#pragma once

#include "search.hpp"

namespace wsp {

constexpr int kOpChunk = 2048;     // products per workgroup (its partial C)
constexpr int kOpBlock = 1024;     // threads of the expand kernel
constexpr int kOpStage = 1024;     // k indices a chunk stages in LDS
constexpr int kOpRowCap = 4096;    // longest row bucket sorted whole in LDS; also the run and merge tile length
constexpr int kOpRowBlock = 256;   // threads per long row in the coalesce
constexpr int kOpHugeBlock = 1024; // threads per row past kOpRowCap
constexpr int64_t kOpNoKey = 0x7fffffffffffffffll;

// Products of rank-1 update k: |At_k| * |B_k|.
struct OpProdIn {
    const int32_t *at_rp, *b_rp;
    __device__ __forceinline__ int64_t operator()(int64_t k) const {
        return static_cast<int64_t>(at_rp[k + 1] - at_rp[k]) * static_cast<int64_t>(b_rp[k + 1] - b_rp[k]);
    }
};

// In-place bitonic sort of n (a power of two) key/value pairs in LDS by key,
// ascending, by the threads of the workgroup (all of them call it).
template <typename K>
__device__ void lds_bitonic(K *key, double *val, int n) {
    for (int k = 2; k <= n; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = threadIdx.x; t < (n >> 1); t += blockDim.x) {
                const int i = ((t & ~(j - 1)) << 1) | (t & (j - 1));   // i has bit j clear
                const int p = i + j;
                const bool up = (i & k) == 0;
                const K a = key[i], b = key[p];
                if ((a > b) == up) {
                    key[i] = b;
                    key[p] = a;
                    const double v = val[i];
                    val[i] = val[p];
                    val[p] = v;
                }
            }
            __syncthreads();
        }
    }
}

// Exclusive workgroup scan of one int per thread; *total gets the sum. All
// threads call it; `scratch` holds one int per wave.
__device__ __forceinline__ int block_excl_scan(int x, int *scratch, int *total) {
    const int nw = blockDim.x / kWave;
    const int w = threadIdx.x / kWave;
    const int incl = wave_incl_sum(x);
    if (lane_id() == kWave - 1) scratch[w] = incl;
    __syncthreads();
    int before = 0, t = 0;
    for (int i = 0; i < nw; ++i) {
        const int s = scratch[i];
        before += i < w ? s : 0;
        t += s;
    }
    __syncthreads();
    *total = t;
    return before + incl - x;
}

// 1. A workgroup's partial C: products [q0, q0 + kOpChunk) formed, sorted by
// key = row << 32 | column (row-major order), equal keys summed; written compacted at part_*[q0..)
// with their count in part_len[chunk]; row_cnt[row] counts the entries each
// row receives from all partial Cs (one atomic per run of a row in the
// partial C, which its sort made contiguous).
template <typename V>
__global__ void __launch_bounds__(kOpBlock) op_expand(const int32_t *__restrict__ at_rp,
                                                      const int32_t *__restrict__ at_col,
                                                      const V *__restrict__ at_val,
                                                      const int32_t *__restrict__ b_rp,
                                                      const int32_t *__restrict__ b_col,
                                                      const V *__restrict__ b_val, int K,
                                                      const int64_t *__restrict__ pref, int64_t P,
                                                      int64_t *__restrict__ part_key, double *__restrict__ part_val,
                                                      int32_t *__restrict__ part_len, int32_t *__restrict__ row_cnt) {
    __shared__ int64_t s_key[kOpChunk];
    __shared__ double s_val[kOpChunk];
    __shared__ int64_t c_key[kOpChunk];   // the partial C, compacted
    __shared__ double c_val[kOpChunk];
    __shared__ int64_t s_pref[kOpStage];
    __shared__ int s_t[2];
    __shared__ int s_scan[kOpBlock / kWave];
    const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kOpChunk;
    if (q0 >= P) return;   // whole workgroup
    const int64_t q1 = P - q0 < kOpChunk ? P : q0 + kOpChunk;
    if (threadIdx.x < kWave) {
        const int t0 = wave_find_entry(pref, K, q0);
        const int t1 = wave_find_entry(pref, K, q1 - 1);
        if (threadIdx.x == 0) {
            s_t[0] = t0;
            s_t[1] = t1;
        }
    }
    __syncthreads();
    const int t0 = s_t[0];
    const int nt = s_t[1] - t0 + 1;
    const bool staged = nt <= kOpStage;
    if (staged)
        for (int k = threadIdx.x; k < nt; k += blockDim.x) s_pref[k] = pref[t0 + k];
    __syncthreads();
    for (int s = threadIdx.x; s < kOpChunk; s += blockDim.x) {
        const int64_t q = q0 + s;
        int64_t key = kOpNoKey;
        double v = 0.0;
        if (q < q1) {
            const int k = staged ? t0 + lds_find_entry(s_pref, nt, q) : t0 + lds_find_entry(pref + t0, nt, q);
            const int64_t r = q - (staged ? s_pref[k - t0] : pref[k]);
            const int64_t nb = b_rp[k + 1] - b_rp[k];   // > 0: index k has products
            const int64_t ai = r / nb;
            const int ia = at_rp[k] + static_cast<int>(ai);
            const int jb = b_rp[k] + static_cast<int>(r - ai * nb);
            key = static_cast<int64_t>(at_col[ia]) << 32 | static_cast<uint32_t>(b_col[jb]);
            v = to_d(at_val[ia]) * to_d(b_val[jb]);
        }
        s_key[s] = key;
        s_val[s] = v;
    }
    __syncthreads();
    lds_bitonic(s_key, s_val, kOpChunk);
    // heads of runs of equal keys, two slots per thread
    constexpr int PER = kOpChunk / kOpBlock;
    int heads = 0;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int s = threadIdx.x * PER + u;
        const int64_t kk = s_key[s];
        heads += (kk != kOpNoKey && (s == 0 || s_key[s - 1] != kk)) ? 1 : 0;
    }
    int total = 0;
    int pos = block_excl_scan(heads, s_scan, &total);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int s = threadIdx.x * PER + u;
        const int64_t kk = s_key[s];
        if (kk == kOpNoKey || (s > 0 && s_key[s - 1] == kk)) continue;
        double sum = s_val[s];
        for (int e = s + 1; e < kOpChunk && s_key[e] == kk; ++e) sum += s_val[e];
        c_key[pos] = kk;
        c_val[pos] = sum;
        ++pos;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < total; t += blockDim.x) {
        const int64_t kk = c_key[t];
        part_key[q0 + t] = kk;
        part_val[q0 + t] = c_val[t];
        const int64_t row = kk >> 32;
        if (t == 0 || (c_key[t - 1] >> 32) != row) {
            int e = t + 1;
            while (e < total && (c_key[e] >> 32) == row) ++e;
            atomicAdd(&row_cnt[row], e - t);
        }
    }
    if (threadIdx.x == 0) part_len[blockIdx.x] = total;
}

// 2a. Each run of a row in a partial C claims that many slots of the row's
// bucket (one atomic) and copies its entries there.
__global__ void __launch_bounds__(256) op_bucket(const int64_t *__restrict__ part_key,
                                                 const double *__restrict__ part_val,
                                                 const int32_t *__restrict__ part_len,
                                                 const int64_t *__restrict__ bucket_off, int32_t *__restrict__ row_fill,
                                                 int32_t *__restrict__ bkt_col, double *__restrict__ bkt_val) {
    __shared__ int32_t s_row[kOpChunk];
    const int len = part_len[blockIdx.x];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kOpChunk;
    for (int t = threadIdx.x; t < len; t += blockDim.x) s_row[t] = static_cast<int32_t>(part_key[base + t] >> 32);
    __syncthreads();
    for (int t = threadIdx.x; t < len; t += blockDim.x) {
        const int row = s_row[t];
        if (t > 0 && s_row[t - 1] == row) continue;
        int e = t + 1;
        while (e < len && s_row[e] == row) ++e;
        const int64_t pos = bucket_off[row] + atomicAdd(&row_fill[row], e - t);
        for (int u = t; u < e; ++u) {
            bkt_col[pos + (u - t)] = static_cast<int32_t>(part_key[base + u] & 0xffffffffll);
            bkt_val[pos + (u - t)] = part_val[base + u];
        }
    }
}

// 2b. Short buckets, S lanes per row (S = 32: buckets of at most 32 entries;
// S = 64: 33 to 64, and the longer ones are listed: up to kOpRowCap from the
// front of long_rows for op_merge_long (count in counters[0]), the rest from
// its back for op_merge_huge (count in counters[2])): sorted in registers
// (bitonic through lane shuffles within the S-lane group), equal columns
// summed, written back compacted from the bucket's start (columns in bkt_col,
// values rounded to V in out_val).

template <int S, typename V>
__global__ void __launch_bounds__(256) op_merge_short(const int64_t *__restrict__ bucket_off, int64_t m,
                                                      int32_t *__restrict__ bkt_col,
                                                      const double *__restrict__ bkt_val, V *__restrict__ out_val,
                                                      int32_t *__restrict__ row_nnz, int32_t *__restrict__ long_rows,
                                                      int32_t *counters) {
    static_assert(S == 32 || S == 64, "groups of 32 or 64 lanes");
    const int64_t row = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) / S;
    const int ln = lane_id() % S;
    const int64_t lo = row < m ? bucket_off[row] : 0;
    const int64_t len = row < m ? bucket_off[row + 1] - lo : 0;
    // this kernel's rows: lengths (S/2, S] (and 0 .. S/2 too when S = 32)
    const bool mine = row < m && len <= S && (S == 32 || len > S / 2);
    if (S == 64 && row < m && len > S && ln == 0) {
        if (len > kOpRowCap)
            long_rows[m - 1 - atomicAdd(&counters[2], 1)] = static_cast<int32_t>(row);
        else
            long_rows[atomicAdd(&counters[0], 1)] = static_cast<int32_t>(row);
    }
    // a wave without a row of this kernel is done; in the others every group takes part in the shuffles
    if (ballot(mine) == 0ull) return;
    int key = mine && ln < len ? bkt_col[lo + ln] : 0x7fffffff;
    double v = mine && ln < len ? bkt_val[lo + ln] : 0.0;
    for (int k = 2; k <= S; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int ok = __shfl_xor(key, j, S);
            const double ov = __shfl_xor(v, j, S);
            const bool lower = (ln & j) == 0;
            const bool up = (ln & k) == 0;
            // the lower lane of an ascending pair keeps the smaller key
            const bool take = lower == up ? ok < key : ok > key;
            if (take) {
                key = ok;
                v = ov;
            }
        }
    }
    const int prev = __shfl_up(key, 1, S);
    const bool head = mine && ln < len && (ln == 0 || prev != key);
    const uint64_t hw = ballot(head);
    const int gbase = lane_id() - ln;   // the group's first lane in the wave
    const uint64_t hm = S == 64 ? hw : (hw >> gbase) & 0xffffffffull;
    // sum each run: a head adds the values of the lanes after it with its key
    double sum = v;
    for (int d = 1; d < S; ++d) {
        const int ok = __shfl_down(key, d, S);
        const double ov = __shfl_down(v, d, S);
        const bool more = ln + d < len && ok == key;
        if (ballot(head && more) == 0ull) break;
        if (head && more) sum += ov;
    }
    if (head) {
        const int pos = __popcll(hm & ((1ull << ln) - 1ull));
        bkt_col[lo + pos] = key;
        out_val[lo + pos] = static_cast<V>(sum);
    }
    if (mine && ln == 0) row_nnz[row] = __popcll(hm);
}

// 2c. Long buckets (65 .. kOpRowCap entries), a workgroup per row, rows taken
// grid-stride from the list op_merge_short made: the bucket is sorted in LDS
// and compacted as in op_merge_short.
template <typename V>
__global__ void __launch_bounds__(kOpRowBlock) op_merge_long(const int64_t *__restrict__ bucket_off,
                                                             int32_t *__restrict__ bkt_col,
                                                             const double *__restrict__ bkt_val,
                                                             V *__restrict__ out_val, int32_t *__restrict__ row_nnz,
                                                             const int32_t *__restrict__ long_rows,
                                                             const int32_t *counters) {
    __shared__ int32_t s_key[kOpRowCap];
    __shared__ double s_val[kOpRowCap];
    __shared__ int s_scan[kOpRowBlock / kWave];
    constexpr int PER = kOpRowCap / kOpRowBlock;
    const int nrows = counters[0];
    for (int idx = blockIdx.x; idx < nrows; idx += gridDim.x) {
        const int row = long_rows[idx];
        const int64_t lo = bucket_off[row];
        const int len = static_cast<int>(bucket_off[row + 1] - lo);
        int np = kWave * 2;
        while (np < len) np <<= 1;
        for (int s = threadIdx.x; s < np; s += blockDim.x) {
            s_key[s] = s < len ? bkt_col[lo + s] : 0x7fffffff;
            s_val[s] = s < len ? bkt_val[lo + s] : 0.0;
        }
        __syncthreads();
        lds_bitonic(s_key, s_val, np);
        int heads = 0;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int s = threadIdx.x * PER + u;
            heads += (s < len && (s == 0 || s_key[s - 1] != s_key[s])) ? 1 : 0;
        }
        int total = 0;
        int pos = block_excl_scan(heads, s_scan, &total);
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int s = threadIdx.x * PER + u;
            if (s >= len || (s > 0 && s_key[s - 1] == s_key[s])) continue;
            const int kk = s_key[s];
            double sum = s_val[s];
            for (int e = s + 1; e < len && s_key[e] == kk; ++e) sum += s_val[e];
            bkt_col[lo + pos] = kk;
            out_val[lo + pos] = static_cast<V>(sum);
            ++pos;
        }
        if (threadIdx.x == 0) row_nnz[row] = total;
        __syncthreads();   // LDS is reused by the next row
    }
}

__device__ __forceinline__ int lds_lower_bound(const int32_t *k, int n, int32_t key) {
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (k[mid] < key) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ int lds_upper_bound(const int32_t *k, int n, int32_t key) {
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (k[mid] <= key) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// 2d. Buckets longer than kOpRowCap, a workgroup per row, rows taken
// grid-stride from the back of long_rows (op_merge_short lists them there):
//   runs of kOpRowCap entries are sorted in LDS into buffer X; then runs are
//   merged pairwise, X to Y and back, doubling their length until one is left:
//   each output tile of kOpRowCap entries takes its share of the two runs
//   (merge-path splits at its ends), merges it in LDS by ranks and writes it
//   out coalesced; last, the sorted row is compacted into the bucket's start
//   as in the shorter tiers. X and Y hold a column array and a value array
//   each, indexed like the bucket; y_val is bkt_val itself (the first step has
//   read the row's bucket before the first merge overwrites it).
template <typename V>
__global__ void __launch_bounds__(kOpHugeBlock) op_merge_huge(const int64_t *__restrict__ bucket_off, int64_t m,
                                                              int32_t *bkt_col, double *bkt_val, V *out_val,
                                                              int32_t *__restrict__ row_nnz,
                                                              const int32_t *__restrict__ long_rows,
                                                              const int32_t *counters, int32_t *x_col, double *x_val,
                                                              int32_t *y_col) {
    __shared__ int32_t s_key[kOpRowCap];
    __shared__ double s_val[kOpRowCap];
    __shared__ int32_t o_key[kOpRowCap];
    __shared__ double o_val[kOpRowCap];
    __shared__ int64_t s_split[2];
    __shared__ int s_scan[kOpHugeBlock / kWave];
    const int nrows = counters[2];
    for (int idx = blockIdx.x; idx < nrows; idx += gridDim.x) {
        const int row = long_rows[m - 1 - idx];
        const int64_t lo = bucket_off[row];
        const int64_t len = bucket_off[row + 1] - lo;
        // runs sorted in LDS, bucket -> X
        for (int64_t r0 = 0; r0 < len; r0 += kOpRowCap) {
            const int n = static_cast<int>(len - r0 < kOpRowCap ? len - r0 : kOpRowCap);
            int np = kWave * 2;
            while (np < n) np <<= 1;
            for (int e = threadIdx.x; e < np; e += blockDim.x) {
                s_key[e] = e < n ? bkt_col[lo + r0 + e] : 0x7fffffff;
                s_val[e] = e < n ? bkt_val[lo + r0 + e] : 0.0;
            }
            __syncthreads();
            lds_bitonic(s_key, s_val, np);
            for (int e = threadIdx.x; e < n; e += blockDim.x) {
                x_col[lo + r0 + e] = s_key[e];
                x_val[lo + r0 + e] = s_val[e];
            }
            __syncthreads();
        }
        // pairwise merges, ping-pong between X and Y
        int32_t *sc = x_col, *dc = y_col;
        double *sv = x_val, *dv = bkt_val;
        for (int64_t w = kOpRowCap; w < len; w <<= 1) {
            for (int64_t s = 0; s < len; s += 2 * w) {
                const int64_t na = len - s < w ? len - s : w;
                const int64_t nb = len - s - na < w ? len - s - na : w;
                const int32_t *ak = sc + lo + s, *bk = ak + na;
                const double *av = sv + lo + s, *bv = av + na;
                for (int64_t d0 = 0; d0 < na + nb; d0 += kOpRowCap) {
                    const int64_t d1 = na + nb - d0 < kOpRowCap ? na + nb : d0 + kOpRowCap;
                    if (threadIdx.x < 2 * kWave) {
                        const int64_t i = wave_merge_split(ak, na, bk, nb, threadIdx.x < kWave ? d0 : d1);
                        if (lane_id() == 0) s_split[threadIdx.x / kWave] = i;
                    }
                    __syncthreads();
                    const int64_t i0 = s_split[0], i1 = s_split[1];
                    const int sa = static_cast<int>(i1 - i0), nt = static_cast<int>(d1 - d0);
                    const int64_t j0 = d0 - i0;
                    for (int e = threadIdx.x; e < nt; e += blockDim.x) {
                        s_key[e] = e < sa ? ak[i0 + e] : bk[j0 + (e - sa)];
                        s_val[e] = e < sa ? av[i0 + e] : bv[j0 + (e - sa)];
                    }
                    __syncthreads();
                    for (int e = threadIdx.x; e < nt; e += blockDim.x) {
                        const int32_t key = s_key[e];
                        const int pos = e < sa ? e + lds_lower_bound(s_key + sa, nt - sa, key)
                                               : (e - sa) + lds_upper_bound(s_key, sa, key);
                        o_key[pos] = key;
                        o_val[pos] = s_val[e];
                    }
                    __syncthreads();
                    for (int e = threadIdx.x; e < nt; e += blockDim.x) {
                        dc[lo + s + d0 + e] = o_key[e];
                        dv[lo + s + d0 + e] = o_val[e];
                    }
                    __syncthreads();   // s_split and the LDS tiles are reused
                }
            }
            int32_t *tc = sc;
            sc = dc;
            dc = tc;
            double *tv = sv;
            sv = dv;
            dv = tv;
        }
        // compaction of the sorted row (sc, sv) into the bucket's start
        int64_t base = 0;
        for (int64_t e0 = 0; e0 < len; e0 += blockDim.x) {
            const int64_t e = e0 + threadIdx.x;
            const int32_t key = e < len ? sc[lo + e] : 0;
            const bool head = e < len && (e == 0 || sc[lo + e - 1] != key);
            int total = 0;
            const int pos = block_excl_scan(head ? 1 : 0, s_scan, &total);
            if (head) {
                double sum = 0.0;
                for (int64_t f = e; f < len && sc[lo + f] == key; ++f) sum += sv[lo + f];
                bkt_col[lo + base + pos] = key;
                out_val[lo + base + pos] = static_cast<V>(sum);
            }
            base += total;
        }
        if (threadIdx.x == 0) row_nnz[row] = static_cast<int32_t>(base);
        __syncthreads();   // LDS is reused by the next row
    }
}

}  // namespace wsp
