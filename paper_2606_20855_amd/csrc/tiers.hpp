// The four row tiers of the symbolic and numeric phases.
//
// Every tier computes, for each of its rows i, the Gustavson accumulation of
// the paper's SpGEMM program (Section 5.1): w[j] += A[i,k] * B[k,j] over the
// entries of row i of A and of row k of B, then copies w into row i of C in
// increasing column order. Products are formed in double and accumulated in
// double for both value types; float outputs are rounded once when written.
// The tiers differ only in where the workspace w lives:
//   tiny  - in registers of one wave segment (products sorted, then reduced)
//   hash  - an LDS open-addressing hash table per row
//   dense - an LDS bitmap over all columns (symbolic) or a dense LDS window of
//           columns swept across the row (numeric)
//   spill - a global-memory hash table from a bounded pool (long rows)
// Rows are independent: each row of C is written only by the threads that own
// it, so no synchronization crosses rows.
#pragma once

#include "device_common.hpp"

namespace wsp {

struct BRowRange {
    const int32_t *b_rp;
    __device__ __forceinline__ int2 operator()(int32_t k) const {
        return make_int2(b_rp[k], b_rp[k + 1]);
    }
};

// Slice of B row k covering column windows [w, w_end) (w_end = w + 1 by
// default), from the window table.
struct BWindowRange {
    const int32_t *wtab;
    int64_t stride;
    int w;
    int w_end = -1;
    __device__ __forceinline__ int2 operator()(int32_t k) const {
        const int32_t *t = wtab + static_cast<int64_t>(k) * stride;
        return make_int2(t[w], t[w_end < 0 ? w + 1 : w_end]);
    }
};

template <typename V>
struct Mats {
    const int32_t *a_rp, *a_col;
    const V *a_val;
    const int32_t *b_rp, *b_col;
    const V *b_val;
};

// ---------------------------------------------------------------------------
// Tiny tier: rows with at most S products, one aligned segment of S lanes per
// row. Lane l of the segment fetches product l into registers; the segment
// bitonic-sorts (column, product) pairs with lane shuffles, sums runs of equal
// columns with a segmented scan, and the last lane of each run emits.
// ---------------------------------------------------------------------------
template <int S, typename V, bool NUM>
__global__ void __launch_bounds__(256) tiny_kernel(Mats<V> M, const int32_t *__restrict__ rows,
                                                   int32_t nrows, int32_t *__restrict__ row_nnz, RowSink out,
                                                   int32_t *__restrict__ c_col, V *__restrict__ c_val,
                                                   Control *ctrl) {
    constexpr int G = 256 / S;
    const int ln = lane_id();
    const int sl = ln & (S - 1);
    const int gidx = blockIdx.x * G + static_cast<int>(threadIdx.x) / S;
    if (gidx >= nrows) return;   // whole segment leaves together
    const int row = rows[gidx];
    const int a_lo = M.a_rp[row], a_hi = M.a_rp[row + 1];

    int key = kPadKey;
    double val = 0.0;
    int base = 0;
    for (int a0 = a_lo; a0 < a_hi; a0 += S) {
        const int a = a0 + sl;
        int bs = 0, len = 0;
        double av = 0.0;
        if (a < a_hi) {
            const int32_t k = M.a_col[a];
            bs = M.b_rp[k];
            len = M.b_rp[k + 1] - bs;
            if (NUM) av = to_d(M.a_val[a]);
        }
        const int incl = group_incl_scan<S>(len);
        const int tot = __shfl(incl, S - 1, S);
        if (tot > 0) {
            const int p = sl - base;
            const int q = p < 0 ? 0 : (p < tot ? p : tot - 1);
            const int o = group_count_le<S>(incl, q);
            const int bs_o = __shfl(bs, o, S);
            const int ex_o = __shfl(incl - len, o, S);
            double av_o = 0.0;
            if (NUM) av_o = __shfl(av, o, S);
            if (p >= 0 && p < tot) {
                const int b = bs_o + (q - ex_o);
                key = M.b_col[b];
                if (NUM) val = av_o * to_d(M.b_val[b]);
            }
            base += tot;
        }
    }

    // bitonic sort of the segment by column
#pragma unroll
    for (int k = 2; k <= S; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int ok = __shfl_xor(key, j, S);
            double ov = 0.0;
            if (NUM) ov = __shfl_xor(val, j, S);
            const bool up = (sl & k) == 0;
            const bool lower = (sl & j) == 0;
            const bool take = (lower == up) ? (ok < key) : (ok > key);
            if (take) {
                key = ok;
                if (NUM) val = ov;
            }
        }
    }

    const int prv = __shfl_up(key, 1, S);
    const int nxt = __shfl_down(key, 1, S);
    if (NUM) {
        // segmented inclusive sum over runs of equal keys
        int start = (sl == 0 || prv != key) ? sl : 0;
#pragma unroll
        for (int o = 1; o < S; o <<= 1) {
            const int y = __shfl_up(start, o, S);
            if (sl >= o) start = start > y ? start : y;
        }
#pragma unroll
        for (int o = 1; o < S; o <<= 1) {
            const double y = __shfl_up(val, o, S);
            if (sl - o >= start) val += y;
        }
    }
    const bool tail = key != kPadKey && (sl == S - 1 || nxt != key);
    const uint64_t bal = ballot(tail);
    const int gbase = ln & ~(S - 1);
    const uint64_t gmask = (S == 64) ? ~0ull : (((1ull << S) - 1ull) << gbase);
    const uint64_t mine = bal & gmask;
    const int count = __popcll(mine);
    if (!NUM) {
        if (sl == 0) row_nnz[row] = count;
        return;
    }
    const int rank = __popcll(mine & ((1ull << ln) - 1ull));
    int64_t cb, seg;
    if (!out.pooled()) {
        cb = out.c_rp[row];
        seg = out.c_rp[row + 1] - cb;
        if (sl == 0 && count != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
    } else {
        int64_t b = 0, l = 0;
        if (sl == 0) b = out.claim(row, count, &l);
        cb = shfl_i64(b, 0, S);
        seg = shfl_i64(l, 0, S);
    }
    if (tail && rank < seg) {
        c_col[cb + rank] = key;
        c_val[cb + rank] = static_cast<V>(val);
    }
}

// ---------------------------------------------------------------------------
// LDS hash table helpers.
// ---------------------------------------------------------------------------

// Adds `prod` at key `col` of an LDS open-addressing table of 2^log2t slots
// (Fibonacci hash, linear probing). Returns 1 if the key was new, 0 if it was
// already present, -1 if every slot was probed without finding room.
template <bool NUM>
__device__ __forceinline__ int lds_insert(int32_t *keys, double *vals, int log2t, int col, double prod) {
    const uint32_t mask = (1u << log2t) - 1u;
    uint32_t h = hash_slot(col, log2t);
    for (uint32_t probe = 0; probe <= mask; ++probe) {
        // one compare-and-swap per probe: it claims an empty slot or reports the key that holds it
        const int old = atomicCAS(&keys[h], kEmptyKey, col);
        if (old == kEmptyKey || old == col) {
            if (NUM) atomicAdd(&vals[h], prod);
            return old == kEmptyKey ? 1 : 0;
        }
        h = (h + 1) & mask;
    }
    return -1;
}

// Writes the occupied slots of an LDS hash table (keys[0..T), vals[0..T)) to
// C[cb + out0 ...] in increasing column order without sorting them. Columns
// [col_lo, col_hi) are covered in bitmap windows of BWW*32 columns: the table's
// columns are marked in an LDS presence bitmap, words are grouped by eight
// and the groups' exclusive prefix counts taken, and every entry's position is
// its group's offset plus the set bits before it in its group. Writes never
// reach past C[cb + seg). Returns the new output count (uniform).
template <int BLOCK, int BWW, typename V>
__device__ int64_t rank_emit(const int32_t *keys, const double *vals, int T, int64_t col_lo, int64_t col_hi,
                             uint32_t *bm, int32_t *goff, int32_t *scratch, int32_t *__restrict__ c_col,
                             V *__restrict__ c_val, int64_t cb, int64_t out0, int64_t seg) {
    constexpr int64_t SPAN = int64_t(BWW) * 32;
    int64_t out = out0;
    for (int64_t wb = col_lo; wb < col_hi; wb += SPAN) {
        const int span = static_cast<int>((col_hi - wb) < SPAN ? (col_hi - wb) : SPAN);
        const int ngroups = (span + 255) >> 8;
        for (int i = threadIdx.x; i < ngroups * 8; i += BLOCK) bm[i] = 0u;
        __syncthreads();
        for (int s = threadIdx.x; s < T; s += BLOCK) {
            const int k = keys[s];
            if (k != kEmptyKey && k >= wb && k < wb + span) {
                const int rel = static_cast<int>(k - wb);
                atomicOr(&bm[rel >> 5], 1u << (rel & 31));
            }
        }
        __syncthreads();
        int carry = 0;
        for (int g0 = 0; g0 < ngroups; g0 += BLOCK) {
            const int g = g0 + threadIdx.x;
            int cnt = 0;
            if (g < ngroups) {
#pragma unroll
                for (int i = 0; i < 8; ++i) cnt += __popc(bm[g * 8 + i]);
            }
            int tot;
            const int ex = block_excl_scan<BLOCK>(cnt, &tot, scratch);
            if (g < ngroups) goff[g] = carry + ex;
            carry += tot;
        }
        __syncthreads();
        for (int s = threadIdx.x; s < T; s += BLOCK) {
            const int k = keys[s];
            if (k != kEmptyKey && k >= wb && k < wb + span) {
                const int rel = static_cast<int>(k - wb);
                const int word = rel >> 5;
                int r = goff[word >> 3];
                for (int i = word & ~7; i < word; ++i) r += __popc(bm[i]);
                r += __popc(bm[word] & ((1u << (rel & 31)) - 1u));
                const int64_t pos = out + r;
                if (pos < seg) {
                    c_col[cb + pos] = k;
                    c_val[cb + pos] = static_cast<V>(vals[s]);
                }
            }
        }
        out += carry;
        __syncthreads();
    }
    return out;
}

// Writes the entries a workgroup holds in registers (thread t: keys kk[j] and
// sums vv[j], kEmptyKey where none) to C[cb + ...] in increasing column order
// without sorting them. The columns [0, ncols) are covered in windows of BWW*32
// columns; for each, the window's keys are marked in a presence bitmap, the
// words are grouped by eight, the groups' exclusive prefix counts are taken,
// and every entry's position is its group's offset plus the set bits before it
// in its group. bm holds BWW words (16-byte aligned) and goff BWW/8 ints. Writes
// never reach past C[cb + seg). Returns the number of entries (uniform).
template <int BLOCK, int BWW, int PER, typename V>
__device__ int64_t rank_emit_regs(const int32_t (&kk)[PER], const double (&vv)[PER], int64_t ncols, uint32_t *bm,
                                  int32_t *goff, int32_t *scratch, int32_t *__restrict__ c_col,
                                  V *__restrict__ c_val, int64_t cb, int64_t seg) {
    constexpr int64_t SPAN = int64_t(BWW) * 32;
    static_assert(BWW % 8 == 0, "whole groups of eight words");
    int64_t out = 0;
    for (int64_t wb = 0; wb < ncols; wb += SPAN) {
        const int span = static_cast<int>((ncols - wb) < SPAN ? (ncols - wb) : SPAN);
        const int ngroups = (span + 255) >> 8;
        for (int i = threadIdx.x; i < ngroups * 8; i += BLOCK) bm[i] = 0u;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int k = kk[j];
            if (k != kEmptyKey && k >= wb && k - wb < span) {
                const int rel = static_cast<int>(k - wb);
                atomicOr(&bm[rel >> 5], 1u << (rel & 31));
            }
        }
        __syncthreads();
        int carry = 0;
        for (int g0 = 0; g0 < ngroups; g0 += BLOCK) {
            const int g = g0 + threadIdx.x;
            int cnt = 0;
            if (g < ngroups) {
                const uint4 lo = reinterpret_cast<const uint4 *>(bm)[2 * g];
                const uint4 hi = reinterpret_cast<const uint4 *>(bm)[2 * g + 1];
                cnt = __popc(lo.x) + __popc(lo.y) + __popc(lo.z) + __popc(lo.w) + __popc(hi.x) + __popc(hi.y) +
                      __popc(hi.z) + __popc(hi.w);
            }
            int tot;
            const int ex = block_excl_scan<BLOCK>(cnt, &tot, scratch);
            if (g < ngroups) goff[g] = carry + ex;
            carry += tot;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int k = kk[j];
            if (k != kEmptyKey && k >= wb && k - wb < span) {
                const int rel = static_cast<int>(k - wb);
                const int word = rel >> 5;
                const uint4 lo = reinterpret_cast<const uint4 *>(bm)[(word >> 3) * 2];
                const uint4 hi = reinterpret_cast<const uint4 *>(bm)[(word >> 3) * 2 + 1];
                const uint32_t w8[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
                const int wi = word & 7;
                int r = goff[word >> 3];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const uint32_t m = i < wi ? 0xffffffffu : (i == wi ? (1u << (rel & 31)) - 1u : 0u);
                    r += __popc(w8[i] & m);
                }
                const int64_t pos = out + r;
                if (pos < seg) {
                    c_col[cb + pos] = k;
                    c_val[cb + pos] = static_cast<V>(vv[j]);
                }
            }
        }
        out += carry;
        __syncthreads();
    }
    return out;
}

// Writes the entries a workgroup holds in registers (thread t: keys kk[j] and
// sums vv[j], kEmptyKey where none; distinct columns) to C[cb + ...] in
// increasing column order, at a cost that follows the entries, not the column
// range. The columns are cut into nb buckets of W = 2^sh columns; each entry
// counts itself into its bucket (an LDS atomic that also gives it a place in
// the bucket); one exclusive scan gives every bucket its first output position
// and numbers the heavy buckets (more than H = max(8, W/16) entries); the
// entries are staged bucket by bucket. An entry's position is its bucket's
// first plus its rank in the bucket: in a light bucket, the staged entries
// with a smaller column (at most H to compare); in a heavy bucket, the set
// bits below it in the bucket's own bitmap of W bits (heavy buckets number at
// most entries / H, so their bitmaps take at most half an int per entry).
// mem holds nb + 1 ints of counts and then the heavy buckets' bitmaps; stage
// one int per entry. Entries number at most 65535. Writes never reach past
// C[cb + seg). Returns the number of entries (uniform).
template <int BLOCK, int PER, typename V>
__device__ int64_t bucket_emit_regs(const int32_t (&kk)[PER], const double (&vv)[PER], int sh, int nb,
                                    int32_t *mem, int32_t *stage, int32_t *scratch, int32_t *__restrict__ c_col,
                                    V *__restrict__ c_val, int64_t cb, int64_t seg) {
    int32_t *cnt = mem;
    uint32_t *bm = reinterpret_cast<uint32_t *>(mem + nb + 1);
    const int W = 1 << sh;
    const int WB = W > 32 ? W >> 5 : 1;   // bitmap words per heavy bucket
    const int H = W / 16 > 8 ? W / 16 : 8;
    for (int i = threadIdx.x; i <= nb; i += BLOCK) cnt[i] = 0;
    __syncthreads();
    int q[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) q[j] = kk[j] != kEmptyKey ? atomicAdd(&cnt[kk[j] >> sh], 1) : 0;
    __syncthreads();
    // exclusive scan, in place, of count | (heavy << 16): low half the bucket's first position, high half its
    // heavy-bucket index; cnt[nb] receives the totals
    const int per = (nb + BLOCK - 1) / BLOCK;
    const int b0 = static_cast<int>(threadIdx.x) * per;
    int part = 0;
    for (int i = 0; i < per; ++i) {
        const int c = b0 + i < nb ? cnt[b0 + i] : 0;
        part += c | (c > H ? 1 << 16 : 0);
    }
    int total;
    int run = block_excl_scan<BLOCK>(part, &total, scratch);
    for (int i = 0; i < per; ++i) {
        if (b0 + i < nb) {
            const int c = cnt[b0 + i];
            cnt[b0 + i] = run;
            run += c | (c > H ? 1 << 16 : 0);
        }
    }
    if (threadIdx.x == 0) cnt[nb] = total;
    __syncthreads();
    const int nwords = (total >> 16) * WB;
    for (int i = threadIdx.x; i < nwords; i += BLOCK) bm[i] = 0u;
#pragma unroll
    for (int j = 0; j < PER; ++j)
        if (kk[j] != kEmptyKey) stage[(cnt[kk[j] >> sh] & 0xffff) + q[j]] = kk[j];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int k = kk[j];
        if (k == kEmptyKey) continue;
        const int b = k >> sh;
        const int lo = cnt[b], hi = cnt[b + 1];
        if ((hi & 0xffff) - (lo & 0xffff) > H) {
            const int rel = k - (b << sh);
            atomicOr(&bm[(lo >> 16) * WB + (rel >> 5)], 1u << (rel & 31));
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int k = kk[j];
        if (k == kEmptyKey) continue;
        const int b = k >> sh;
        const int lo = cnt[b], hi = cnt[b + 1];
        const int first = lo & 0xffff, last = hi & 0xffff;
        int r = 0;
        if (last - first > H) {
            const int rel = k - (b << sh);
            const uint32_t *w = bm + (lo >> 16) * WB;
            for (int i = 0; i < (rel >> 5); ++i) r += __popc(w[i]);
            r += __popc(w[rel >> 5] & ((1u << (rel & 31)) - 1u));
        } else {
            for (int i = first; i < last; ++i) r += stage[i] < k;
        }
        const int64_t pos = first + r;
        if (pos < seg) {
            c_col[cb + pos] = k;
            c_val[cb + pos] = static_cast<V>(vv[j]);
        }
    }
    return total & 0xffff;
}

// ---------------------------------------------------------------------------
// Hash tier: one workgroup per row, an LDS table of 2^LOG2T slots.
// Symbolic keeps keys only and counts first insertions. Numeric also adds the
// product into the slot's double, then writes the row in column order, the
// slots moved to registers and the table's memory reused, without a sort:
// tables of 1024 slots and more by rank over a presence bitmap of the columns
// when it takes at most kBitmapEmitMaxWindows windows of the table's memory;
// otherwise tables of 512 slots and more by column buckets (bucket_emit_regs)
// while a bucket spans at most 2^kBucketEmitMaxLog2Width columns, then the
// bitmap again up to kMaxRankWindows windows. Smaller tables, and wider
// column ranges, compact the slots and bitonic-sort them in LDS.
// ---------------------------------------------------------------------------
constexpr int kMaxRankWindows = 4;
constexpr int kBucketEmitMinLog2 = 9;        // tables this large or larger emit by column buckets
constexpr int kBitmapEmitMaxWindows = 2;     // ... unless the column bitmap takes at most this many windows
constexpr int kBucketEmitMaxLog2Width = 9;   // ... while a bucket spans at most 512 columns

template <int LOG2T>
struct HashShape {
    static constexpr int T = 1 << LOG2T;
    static constexpr int BLOCK = T <= 256 ? 64 : (T <= 512 ? 128 : (T <= 2048 ? 256 : (T <= 4096 ? 512 : 1024)));
    // bitmap words for rank emission, held in the T doubles of the table (0: always sort)
    static constexpr int BWW = LOG2T >= 10 ? 2 * T : 0;
};

template <int LOG2T, typename V, bool NUM>
__global__ void __launch_bounds__(HashShape<LOG2T>::BLOCK) hash_kernel(Mats<V> M, const int32_t *__restrict__ rows,
                                                                       int64_t ncols,
                                                                       int32_t *__restrict__ row_nnz, RowSink out,
                                                                       int32_t *__restrict__ c_col,
                                                                       V *__restrict__ c_val, Control *ctrl) {
    constexpr int T = HashShape<LOG2T>::T;
    constexpr int BLOCK = HashShape<LOG2T>::BLOCK;
    constexpr int BWW = NUM ? HashShape<LOG2T>::BWW : 0;
    constexpr int NW = BLOCK / kWave;
    static_assert(T >= BLOCK, "table smaller than block");
    __shared__ int32_t keys[T];
    __shared__ __align__(16) double vals[NUM ? T : 1];
    __shared__ int32_t scratch[NW];
    __shared__ int32_t marks[NW * kMarkInts];
    __shared__ int32_t ctot[kCtotInts];
    __shared__ int64_t s_claim[2];   // pool output: the row's first entry and writable length

    const int row = rows[blockIdx.x];
    for (int i = threadIdx.x; i < T; i += BLOCK) {
        keys[i] = kEmptyKey;
        if (NUM) vals[i] = 0.0;
    }
    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    int32_t *mark = marks + wv * kMarkInts;
    init_marks(mark);
    __syncthreads();

    const int a_lo = M.a_rp[row], a_hi = M.a_rp[row + 1];
    int inserted = 0;
    bool overflow = false;
    for_each_product_wg<BLOCK, V, NUM>(M.a_col, M.a_val, a_lo, a_hi, BRowRange{M.b_rp}, M.b_col, M.b_val, mark,
                                       ctot, [&](int col, double prod) {
                                 const int r = lds_insert<NUM>(keys, vals, LOG2T, col, prod);
                                 inserted += r > 0;
                                 overflow |= r < 0;
                             });
    if (overflow) atomicOr(&ctrl->error_flags, kErrProbeExhausted);

    if (!NUM) {
        const int total = block_sum<BLOCK>(inserted, scratch);
        if (threadIdx.x == 0) row_nnz[row] = total;
        return;
    }
    __syncthreads();

    int64_t cb, seg;
    if (!out.pooled()) {
        cb = out.c_rp[row];
        seg = out.c_rp[row + 1] - cb;
    } else {
        // the row's entries are its first insertions
        const int total = block_sum<BLOCK>(inserted, scratch);
        if (threadIdx.x == 0) s_claim[0] = out.claim(row, total, &s_claim[1]);
        __syncthreads();
        cb = uniform(s_claim[0]);
        seg = uniform(s_claim[1]);
    }
    // the thread's slots, in registers
    constexpr int PER = T / BLOCK;
    int kk[PER];
    double vv[PER];
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int s2 = threadIdx.x + j * BLOCK;
        kk[j] = keys[s2];
        vv[j] = vals[s2];
        cnt += kk[j] != kEmptyKey;
    }
    if constexpr (LOG2T >= kBucketEmitMinLog2) {
        // buckets of 2^sh columns, at most T of them (the doubles' memory holds their counts and the heavy
        // buckets' bitmaps, the keys' the staged entries); where the column range takes at most
        // kBitmapEmitMaxWindows windows of the table's bitmap, rank emission over the bitmap is cheaper
        const int sh = uniform(ceil_log2(ncols) > LOG2T ? ceil_log2(ncols) - LOG2T : 0);
        const int64_t nbw = BWW > 0 ? (ncols + int64_t(BWW) * 32 - 1) / (int64_t(BWW) * 32) : INT64_MAX;
        if (sh <= kBucketEmitMaxLog2Width && nbw > kBitmapEmitMaxWindows) {
            __syncthreads();   // every slot is read: the table's memory takes the counts and the staged keys
            const int nb = static_cast<int>((ncols + (int64_t(1) << sh) - 1) >> sh);
            const int64_t total = bucket_emit_regs<BLOCK, PER, V>(kk, vv, sh, nb, reinterpret_cast<int32_t *>(vals),
                                                                  keys, scratch, c_col, c_val, cb, seg);
            if (threadIdx.x == 0 && !out.pooled() && total != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
            return;
        }
    }
    if constexpr (BWW > 0) {
        const int64_t nbw = (ncols + int64_t(BWW) * 32 - 1) / (int64_t(BWW) * 32);
        if (nbw <= kMaxRankWindows) {
            __syncthreads();   // every slot is read: the table's memory takes the bitmap and the group offsets
            static_assert(BWW <= 2 * T && BWW / 8 <= T, "bitmap in the doubles, group offsets in the keys");
            const int64_t total = rank_emit_regs<BLOCK, BWW, PER, V>(
                kk, vv, ncols, reinterpret_cast<uint32_t *>(vals), keys, scratch, c_col, c_val, cb, seg);
            if (threadIdx.x == 0 && !out.pooled() && total != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
            return;
        }
    }

    // compact occupied slots to the front of the table
    int total;
    int pos = block_excl_scan<BLOCK>(cnt, &total, scratch);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        if (kk[j] != kEmptyKey) {
            keys[pos] = kk[j];
            vals[pos] = vv[j];
            ++pos;
        }
    }
    int n2 = 1;
    while (n2 < total) n2 <<= 1;
    n2 = uniform(n2);
    for (int i = total + threadIdx.x; i < n2; i += BLOCK) keys[i] = kPadKey;
    __syncthreads();

    // bitonic sort of keys[0..n2) (values follow)
    for (int k = 2; k <= n2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < (n2 >> 1); i += BLOCK) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
                const int hi = lo + j;
                const bool up = (lo & k) == 0;
                const int kl = keys[lo], kh = keys[hi];
                if ((kl > kh) == up) {
                    keys[lo] = kh;
                    keys[hi] = kl;
                    const double t = vals[lo];
                    vals[lo] = vals[hi];
                    vals[hi] = t;
                }
            }
            __syncthreads();
        }
    }

    if (threadIdx.x == 0 && !out.pooled() && total != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
    const int lim = static_cast<int64_t>(total) < seg ? total : static_cast<int>(seg);
    for (int i = threadIdx.x; i < lim; i += BLOCK) {
        c_col[cb + i] = keys[i];
        c_val[cb + i] = static_cast<V>(vals[i]);
    }
}

// ---------------------------------------------------------------------------
// Dense tier, symbolic: an LDS bitmap over all NWORDS*32 columns, one
// workgroup per row. The row's entry count is the bitmap's population count.
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Row i of the structure cache (when cache is not null) receives the bitmap
// of the row handled by workgroup i < cache_rows, and slot_of_row[row] = i.
template <int NWORDS, int BLOCK>
__global__ void __launch_bounds__(BLOCK) bitmap_sym_kernel(Mats<float> M,
                                                           const int32_t *__restrict__ rows,
                                                           int nwords_used,
                                                           int32_t *__restrict__ row_nnz,
                                                           int32_t *__restrict__ slot_of_row,
                                                           uint32_t *__restrict__ cache, int64_t row_words,
                                                           int64_t cache_rows) {
    constexpr int NW = BLOCK / kWave;
    __shared__ __align__(16) uint32_t bm[NWORDS];
    __shared__ int32_t scratch[NW];
    __shared__ int32_t marks[NW * kMarkIntsLong];
    __shared__ int32_t ctot[kCtotInts];
    __shared__ int32_t e_col[kCacheEntries], e_bs[kCacheEntries], e_len[kCacheEntries];
    const int row = rows[blockIdx.x];
    static_assert(NWORDS % 4 == 0, "the bitmap is cleared, counted and copied in 16-byte pieces");
    const int nq = (nwords_used + 3) >> 2;   // 16-byte pieces in use (the words past nwords_used stay zero)
    uint4 *const bq = reinterpret_cast<uint4 *>(bm);
    for (int i = threadIdx.x; i < nq; i += BLOCK) bq[i] = make_uint4(0u, 0u, 0u, 0u);
    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    int32_t *mark = marks + wv * kMarkIntsLong;
    init_marks(mark, kMarkIntsLong);
    __syncthreads();
    for_each_product_wg<BLOCK, float, false, true, true>(
        M.a_col, nullptr, M.a_rp[row], M.a_rp[row + 1], BRowRange{M.b_rp}, M.b_col, nullptr, mark, ctot,
        BitmapMark<1>{{}, bm, 0},
        EntryCache{e_col, e_bs, e_len, nullptr, false});
    __syncthreads();
    int cnt = 0;
    const bool caching = cache != nullptr && blockIdx.x < cache_rows;
    uint32_t *const dst = caching ? cache + static_cast<int64_t>(blockIdx.x) * row_words : nullptr;
    for (int i = threadIdx.x; i < nq; i += BLOCK) {
        const uint4 q = bq[i];
        cnt += __popc(q.x) + __popc(q.y) + __popc(q.z) + __popc(q.w);
        // (a cache row holds row_words >= 4 nq words, 16-byte aligned; the words past nwords_used are zero)
        if (caching)
            __builtin_nontemporal_store(u32x4{q.x, q.y, q.z, q.w}, reinterpret_cast<u32x4 *>(dst + 4 * i));
    }
    if (caching && threadIdx.x == 0) slot_of_row[row] = static_cast<int32_t>(blockIdx.x);
    const int total = block_sum<BLOCK>(cnt, scratch);
    if (threadIdx.x == 0) row_nnz[row] = total;
}

// ---------------------------------------------------------------------------
// Dense tier, numeric: the row's columns are swept in windows of WV columns.
// For each window the workgroup accumulates every product whose column falls
// inside it into a dense LDS array of doubles (plus a presence bitmap), then
// emits the window's entries in column order by scanning the bitmap: no hash
// and no sort. Each wave emits its own slice of the window after one barrier
// and clears what it read, so the next window starts from zero. The window
// table gives each B row's slice inside the window.
//
// Because C.row_ptr gives the row's entry count, the kernel knows how many
// entries are still to come after each window. As soon as the remainder fits
// an LDS hash table carved out of the window's own storage, the rest of the
// row (all remaining columns at once) is accumulated in that table and written
// by rank emission. Sparse tails therefore cost one pass instead of one pass
// per window.
// ---------------------------------------------------------------------------
template <int WV>
struct DenseShape {
    // smaller windows use smaller workgroups so more of them share a CU
    static constexpr int BLOCK = WV >= 8192 ? 1024 : (WV >= 4096 ? 512 : 256);
    static constexpr int NW = BLOCK / kWave;
    static constexpr int NWORDS = WV / 32;
    static constexpr int WCOLS = WV / NW;            // columns each wave emits
    static constexpr int TAIL_T = WV / 2;            // tail table slots (12 B each)
    static constexpr int TAIL_LOG2 = WV == 16384 ? 13 : (WV == 8192 ? 12 : (WV == 4096 ? 11 : 9));
    static constexpr int TAIL_CAP = (TAIL_T * 2) / 3;
    static constexpr int BWW = WV / 2;               // tail rank bitmap words
    static_assert(WCOLS % kWave == 0, "window must split into 64-column chunks per wave");
    static_assert(TAIL_T * 12 + BWW * 4 <= WV * 8, "tail table and bitmap must fit in the window");
    static_assert((1 << TAIL_LOG2) == TAIL_T, "tail table size");
};

template <int WV, typename V, bool SENT>
__global__ void __launch_bounds__(DenseShape<WV>::BLOCK) dense_num_kernel(Mats<V> M, const int32_t *__restrict__ rows,
                                                         const int32_t *__restrict__ wtab, int nwin,
                                                         int64_t ncols, const int64_t *__restrict__ c_rp,
                                                         int32_t *__restrict__ c_col,
                                                         V *__restrict__ c_val, Control *ctrl) {
    using S = DenseShape<WV>;
    constexpr int BLOCK = S::BLOCK;
    constexpr int NW = S::NW;
    constexpr int WWORDS = S::WCOLS / 32;
    constexpr int NCH = S::WCOLS / kWave;            // 64-column chunks per wave
    // SENT: slots start at -0.0 and a slot is occupied iff its bits differ
    // from -0.0 (no product is zero, so no sum of products is -0.0); no bitmap.
    constexpr uint64_t kNegZero = 0x8000000000000000ull;
    __shared__ double acc[WV];
    __shared__ uint32_t bm[SENT ? 1 : S::NWORDS];
    __shared__ int32_t wave_cnt[NW];
    __shared__ int32_t goff[S::BWW / 8];
    __shared__ int32_t scratch[NW];
    __shared__ int32_t marks[NW * kMarkInts];
    __shared__ int32_t ctot[kCtotInts];

    const int row = rows[blockIdx.x];
    const int a_lo = M.a_rp[row], a_hi = M.a_rp[row + 1];
    const int64_t cb = c_rp[row];
    const int64_t seg = c_rp[row + 1] - cb;
    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    const int ln = lane_id();
    const int64_t stride = static_cast<int64_t>(nwin) + 1;
    int32_t *mark = marks + wv * kMarkInts;
    init_marks(mark);

    int64_t out = 0;
    int w = 0;
    if (seg > S::TAIL_CAP) {
        for (int i = threadIdx.x; i < WV; i += BLOCK) acc[i] = SENT ? __longlong_as_double(kNegZero) : 0.0;
        if (!SENT)
            for (int i = threadIdx.x; i < S::NWORDS; i += BLOCK) bm[i] = 0u;
    }
    __syncthreads();
    for (; w < nwin && seg - out > S::TAIL_CAP; ++w) {
        const int w0 = w * WV;
        for_each_product_wg<BLOCK, V, true>(M.a_col, M.a_val, a_lo, a_hi, BWindowRange{wtab, stride, w}, M.b_col,
                                            M.b_val, mark, ctot, [&](int col, double prod) {
                                      const int loc = col - w0;
                                      atomicAdd(&acc[loc], prod);
                                      if (!SENT) atomicOr(&bm[loc >> 5], 1u << (loc & 31));
                                  });
        __syncthreads();
        // each wave counts its slice, then emits it at its offset
        const int wbase = wv * S::WCOLS;
        uint64_t occ[NCH];
        int cnt = 0;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int loc = wbase + c * kWave + ln;
            bool set;
            if (SENT) set = static_cast<uint64_t>(__double_as_longlong(acc[loc])) != kNegZero;
            else set = (bm[loc >> 5] >> (loc & 31)) & 1u;
            occ[c] = ballot(set);
            cnt += __popcll(occ[c]);
        }
        if (ln == 0) wave_cnt[wv] = cnt;
        __syncthreads();
        int before = 0, wtot = 0;
        for (int i = 0; i < NW; ++i) {
            const int x = wave_cnt[i];
            before += i < wv ? x : 0;
            wtot += x;
        }
        int64_t pos0 = out + uniform(before);
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int loc = wbase + c * kWave + ln;
            if (occ[c] == 0ull) continue;
            if ((occ[c] >> ln) & 1ull) {
                const int64_t pos = pos0 + __popcll(occ[c] & ((1ull << ln) - 1ull));
                if (pos < seg) {
                    c_col[cb + pos] = w0 + loc;
                    c_val[cb + pos] = static_cast<V>(acc[loc]);
                }
                acc[loc] = SENT ? __longlong_as_double(kNegZero) : 0.0;
            }
            pos0 += __popcll(occ[c]);
        }
        if (!SENT)
            for (int i = ln; i < WWORDS; i += kWave) bm[(wbase >> 5) + i] = 0u;
        out += uniform(wtot);
        __syncthreads();
    }

    if (w < nwin && seg - out > 0) {
        // the remaining columns [w*WV, ncols) fit an LDS hash table
        const int64_t rem = seg - out;
        int log2t = ceil_log2(rem + (rem >> 1));
        if (log2t < 6) log2t = 6;
        log2t = uniform(log2t);
        const int T = 1 << log2t;
        int32_t *tk = reinterpret_cast<int32_t *>(acc);
        double *tv = reinterpret_cast<double *>(tk + T);
        uint32_t *tbm = reinterpret_cast<uint32_t *>(acc) + (2 * WV - S::BWW);
        for (int i = threadIdx.x; i < T; i += BLOCK) {
            tk[i] = kEmptyKey;
            tv[i] = 0.0;
        }
        __syncthreads();
        bool overflow = false;
        for_each_product_wg<BLOCK, V, true>(M.a_col, M.a_val, a_lo, a_hi, BWindowRange{wtab, stride, w, nwin},
                                            M.b_col, M.b_val, mark, ctot, [&](int col, double prod) {
                                      overflow |= lds_insert<true>(tk, tv, log2t, col, prod) < 0;
                                  });
        if (overflow) atomicOr(&ctrl->error_flags, kErrProbeExhausted);
        __syncthreads();
        out = rank_emit<BLOCK, S::BWW, V>(tk, tv, T, static_cast<int64_t>(w) * WV, ncols, tbm, goff, scratch,
                                          c_col, c_val, cb, out, seg);
    }
    if (threadIdx.x == 0 && out != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
}

// ---------------------------------------------------------------------------
// Dense tier, numeric, rank-indexed (default when ncols <= 128 * 8192).
//
// The row is processed in regions of REGION_COLS columns. For a region:
//  1. a structure pass marks every column the row touches in an LDS bitmap;
//  2. each bitmap word gets the exclusive popcount prefix of the words before
//     it, stored beside its bits (one 64-bit LDS read then gives any column's
//     rank among the row's entries in the region);
//  3. the region's ranks are taken in slices of at most CAP entries that end
//     on 8192-column window boundaries where possible; for each slice the
//     values of the products whose columns fall in it are accumulated into a
//     dense LDS array indexed by rank (no hash, no probing), then the slice is
//     staged in rank order (column beside value) and copied to C with
//     coalesced stores.
// Most rows need one region and one or two slices; the accumulator holds
// entries, not columns, so sparse stretches of columns cost nothing. The
// window table (8192-column windows) gives each B row's part inside a range
// of windows.
// ---------------------------------------------------------------------------
constexpr int kRankWinCols = 8192;

// Position of the q-th set bit (counting from 0) of x, for q < popcount(x):
// the largest p whose bits below it number at most q, by binary search (the
// bits below p are a bit-field extract of width p, then a popcount).
__device__ __forceinline__ int select_set_bit(uint32_t x, int q) {
    const uint32_t uq = static_cast<uint32_t>(q);
    int pos = __popc(x & 0xffffu) <= uq ? 16 : 0;
#pragma unroll
    for (int w = 8; w >= 1; w >>= 1) {
        const int t = pos + w;
        pos = static_cast<uint32_t>(__popc(__builtin_amdgcn_ubfe(x, 0u, static_cast<uint32_t>(t)))) <= uq ? t : pos;
    }
    return pos;
}

// Two consecutive values at p (8-byte aligned for float, 16 for double) in
// one streaming store.
typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef double f64x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_pair_nt(int32_t *p, int32_t a, int32_t b) {
    __builtin_nontemporal_store(i32x2{a, b}, reinterpret_cast<i32x2 *>(p));
}
__device__ __forceinline__ void store_pair_nt(float *p, float a, float b) {
    __builtin_nontemporal_store(f32x2{a, b}, reinterpret_cast<f32x2 *>(p));
}
__device__ __forceinline__ void store_pair_nt(double *p, double a, double b) {
    __builtin_nontemporal_store(f64x2{a, b}, reinterpret_cast<f64x2 *>(p));
}

// Marks slot k of the rank kernel's slice with bitmap word wd: the low half of
// the slot's 8-byte accumulator (float output) or the stage array (double).
template <bool PACKED>
__device__ __forceinline__ void rank_mark(double *acc, int32_t *stage, int k, int wd) {
    if constexpr (PACKED) reinterpret_cast<uint2 *>(acc)[k].x = static_cast<uint32_t>(wd);
    else stage[k] = wd;
}

// Shape: 1024 threads, regions of 8192 bitmap words (262144 columns), and a
// rank accumulator of CAP doubles. With float output a staged entry (column,
// value) packs into its own 8-byte accumulator slot; double output stages the
// columns in an array of their own, so its accumulator is smaller.
template <typename V>
struct RankShape {
    static constexpr int BLOCK = 1024;
    static constexpr int REGION_WORDS = 8192;
    static constexpr int REGION_COLS = REGION_WORDS * 32;
    static constexpr int REGION_WINS = REGION_COLS / kRankWinCols;
    static constexpr bool PACKED = sizeof(V) == 4;
    static constexpr int CAP = PACKED ? 10864 : 7232;
    static constexpr int STAGE = PACKED ? 1 : CAP;   // separate column stage (ints)
    static_assert(REGION_COLS % kRankWinCols == 0, "regions hold whole windows");
    static_assert(CAP % 2 == 0, "the copy reads slots in pairs");
    static_assert(REGION_WORDS % (BLOCK / kWave * kWave) == 0, "prefix scan takes whole word rows per wave");
};

// Value visit of the rank kernel: the product's rank among the region's
// entries (bitmap word prefix plus the set bits below it), then an LDS add at
// that rank when it falls in the current slice [r0, r1).
struct RankAccumulate : TwoPhaseVisit {
    const uint2 *bw;
    double *acc;
    int col0, r0, r1;
    // the column's rank relative to r0 (outside [0, r1 - r0) when the slice does not hold it)
    __device__ __forceinline__ int pre(int col) const {
        const int rel = col - col0;
        const uint2 e = bw[rel >> 5];
        // the bits below the column's own: a bit-field extract of width rel mod 32 (the instruction takes the
        // width's low five bits itself)
        return static_cast<int>(e.y) + __popc(__builtin_amdgcn_ubfe(e.x, 0u, static_cast<uint32_t>(rel))) - r0;
    }
    // one unsigned compare keeps the slice's ranks and drops the rest, -1 included
    __device__ __forceinline__ void post(int k, double prod) const {
        if (static_cast<uint32_t>(k) < static_cast<uint32_t>(r1 - r0)) atomicAdd(&acc[k], prod);
    }
    __device__ __forceinline__ int safe_col() const { return col0; }
    __device__ __forceinline__ void operator()(int col, double prod) const { post(pre(col), prod); }
};

// Part of B row k inside the windows [w, w_end) of a rank slice. An entry held
// in the entry cache starts the pass with its slice of the previous pass there
// (for the first pass of a region, the whole region), and its region end in
// e_hi: the new bounds come from those where the slice boundary allows
// (lo_from 0: the previous start, 1: the previous end; hi_from 0: the previous
// end, 1: the region end; 2 for either: the window table), so most passes read
// nothing from memory for the cached entries.
struct SliceRange {
    const int32_t *wtab;
    int64_t stride;
    int w, w_end;
    int lo_from, hi_from;
    const int32_t *e_bs, *e_len, *e_hi;
    __device__ __forceinline__ int2 operator()(int32_t k) const {
        const int32_t *t = wtab + static_cast<int64_t>(k) * stride;
        return make_int2(t[w], t[w_end]);
    }
    __device__ __forceinline__ int2 cached(int32_t k, int ci) const {
        const int bs = e_bs[ci];
        const int be = bs + e_len[ci];
        const int32_t *t = wtab + static_cast<int64_t>(k) * stride;
        const int lo = lo_from == 0 ? bs : lo_from == 1 ? be : t[w];
        const int hi = hi_from == 0 ? be : hi_from == 1 ? e_hi[ci] : t[w_end];
        return make_int2(lo, hi);
    }
};

// A row of the rank kernel, gathered beforehand so that a workgroup fetches
// the next row's description with one load.
struct RankRow {
    int32_t row, a_lo, a_hi;
    int32_t slot;     // the row's structure cache row, or -1
    int64_t cb, seg;  // CSR output: C.row_ptr[row] and the row's entry count
};
static_assert(sizeof(RankRow) == 32, "two 16-byte loads");

__global__ void __launch_bounds__(256) rank_rows(const int32_t *__restrict__ rows, int n,
                                                 const int32_t *__restrict__ a_rp, const int64_t *__restrict__ c_rp,
                                                 const int32_t *__restrict__ slot_of_row, RankRow *__restrict__ out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int row = rows[i];
    RankRow r;
    r.row = row;
    r.a_lo = a_rp[row];
    r.a_hi = a_rp[row + 1];
    r.slot = slot_of_row != nullptr ? slot_of_row[row] : -1;
    r.cb = c_rp != nullptr ? c_rp[row] : 0;
    r.seg = c_rp != nullptr ? c_rp[row + 1] - r.cb : 0;
    out[i] = r;
}

// rank_rows for the dense bins of a binning held on the device (their range of
// perm read from ctrl): the grid covers every row, threads past the dense rows
// do nothing.
__global__ void __launch_bounds__(256) rank_rows_of_bins(const int32_t *__restrict__ perm,
                                                         const Control *__restrict__ ctrl,
                                                         const int32_t *__restrict__ a_rp,
                                                         const int64_t *__restrict__ c_rp,
                                                         const int32_t *__restrict__ slot_of_row,
                                                         RankRow *__restrict__ out) {
    const int start = ctrl->bin_offset[kBinDense0];
    int n = 0;
    for (int b = kBinDense0; b < kBinDense0 + kNumClasses; ++b) n += ctrl->bin_count[b];
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int row = perm[start + i];
    RankRow r;
    r.row = row;
    r.a_lo = a_rp[row];
    r.a_hi = a_rp[row + 1];
    r.slot = slot_of_row[row];
    r.cb = c_rp[row];
    r.seg = c_rp[row + 1] - r.cb;
    out[i] = r;
}

// A zero the compiler cannot see through: an address offset by it is not
// uniform, so the load is a vector load. Prefetches must be vector loads:
// a scalar load counts with the LDS operations, and every barrier and LDS wait
// would then wait for it too.
__device__ __forceinline__ int opaque_zero() {
    int z = 0;
    asm volatile("" : "+v"(z));
    return z;
}

// Rank-indexed dense rows. The grid is persistent (one workgroup per CU, the
// LDS allows no more): workgroups claim rows from a counter in the order of
// `rr` (heaviest first), two rows ahead, and while a row's last slice is staged
// and copied they load the next row's description, its cached bitmap words and
// its entry-cache entries, so a row starts without a round trip to memory.
// When `cache` is not null, a row with slot >= 0 takes its column bitmap from
// that row of the structure cache (written by the symbolic phase for the same
// A and B) instead of running the structure pass.
// POOL selects the output: CSR at C.row_ptr, or pool segments claimed through
// the sink (compiled apart, so the CSR kernel carries none of the pool state).
// OFF32: B's offsets in the value passes' general steps are formed in 32 bits,
// for B with nnz * sizeof(V) <= 2^32 (the launch checks).
template <typename V, bool POOL, bool OFF32>
__global__ void __launch_bounds__(RankShape<V>::BLOCK) dense_rank_kernel(
    Mats<V> M, const RankRow *__restrict__ rr, int nrows, const int32_t *__restrict__ wtab, int nwin, int64_t ncols,
    RowSink out, int32_t *__restrict__ c_col, V *__restrict__ c_val, Control *ctrl,
    const uint32_t *__restrict__ cache, int64_t row_words) {
    using SH = RankShape<V>;
    constexpr int BLOCK = SH::BLOCK;
    constexpr int NW = BLOCK / kWave;
    constexpr int RW = SH::REGION_WORDS;
    constexpr int WROWS = RW / NW / kWave;   // 64-word rows per wave in the prefix scan
    constexpr int WIN_WORDS = kRankWinCols / 32;
    constexpr int CAP = SH::CAP;
    __shared__ uint2 bw[RW];                 // x: column bits, y: exclusive prefix within the region
    __shared__ __align__(16) double acc[CAP];
    __shared__ __align__(16) int32_t stage[SH::STAGE];
    __shared__ int32_t scratch[NW];
    __shared__ int32_t marks[NW * kMarkIntsLong];
    __shared__ int32_t ctot[kCtotInts];
    __shared__ int32_t s_next;   // the claimed next row
    __shared__ int64_t s_claim[2];   // pool output: the row's first entry and writable length
    __shared__ int32_t e_col[kCacheEntries], e_bs[kCacheEntries], e_len[kCacheEntries], e_hi[kCacheEntries];
    __shared__ double e_av[kCacheEntries];

    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    const int ln = lane_id();
    const int64_t stride = static_cast<int64_t>(nwin) + 1;
    const int rg1_first = nwin < SH::REGION_WINS ? nwin : SH::REGION_WINS;   // end of the first region
    int32_t *mark = marks + wv * kMarkIntsLong;
    init_marks(mark, kMarkIntsLong);
    for (int i = threadIdx.x; i < CAP; i += BLOCK) acc[i] = 0.0;
    if constexpr (!SH::PACKED)
        for (int i = threadIdx.x; i < CAP; i += BLOCK) stage[i] = -1;
    if (threadIdx.x == 0) s_next = atomicAdd(&ctrl->rank_next, 1);
    __syncthreads();
    const int idx = uniform(s_next);
    if (idx >= nrows) return;   // the whole workgroup

    // The first region of a cached row, as the row start consumes it: the words this thread scans (wave w owns
    // words [w*RW/NW, (w+1)*RW/NW), one 64-word row at a time) and, for cache entry ci = threadIdx.x, the
    // entry's column, value and part of B in the region. Loaded for the first row here, for later rows while
    // the row before them finishes.
    const int wbase = wv * (RW / NW);
    const int ci = static_cast<int>(threadIdx.x);
    uint32_t bits[WROWS];
    int pk = 0, plo = 0, phi = 0;
    V pav = V(0);   // converted where it is used, so the load need not land before the words' loads go out
    auto fetch_words = [&](int a_lo, int a_hi, int slot) {
        const uint32_t *src = cache + static_cast<int64_t>(slot) * row_words;
        const int nw0 = static_cast<int>((ncols < SH::REGION_COLS ? ncols : SH::REGION_COLS) + 31) >> 5;
        pk = 0;
        pav = V(0);
        if (ci < kCacheEntries && a_lo + ci < a_hi) {
            pk = M.a_col[a_lo + ci];
            pav = M.a_val[a_lo + ci];
        }
#pragma unroll
        for (int q = 0; q < WROWS; ++q) {
            const int i = wbase + q * kWave + ln;
            bits[q] = i < nw0 ? __builtin_nontemporal_load(&src[i]) : 0u;
        }
    };
    auto fetch_bounds = [&](int a_lo, int a_hi) {
        plo = 0;
        phi = 0;
        if (ci < kCacheEntries && a_lo + ci < a_hi) {
            const int32_t *t = wtab + static_cast<int64_t>(pk) * stride;
            plo = t[0];
            phi = t[rg1_first];
        }
    };
    int row = uniform(rr[idx].row), a_lo = uniform(rr[idx].a_lo), a_hi = uniform(rr[idx].a_hi);
    int slot = cache != nullptr ? uniform(rr[idx].slot) : -1;
    int64_t row_cb = POOL ? 0 : uniform(rr[idx].cb), row_seg = POOL ? 0 : uniform(rr[idx].seg);
    if (slot >= 0) {
        fetch_words(a_lo, a_hi, slot);
        fetch_bounds(a_lo, a_hi);
    }
    // thread 0: the row after the next one, claimed a row ahead of its use so that the claim's round trip
    // overlaps a row's work
    int claimed = 0;
    if (threadIdx.x == 0) claimed = atomicAdd(&ctrl->rank_next, 1);
    while (true) {
        // CSR output: the row's place from C.row_ptr. Pool output: claimed once the region's entry count is
        // known
        int64_t cb = row_cb, seg = row_seg;
        EntryCache ecache{e_col, e_bs, e_len, e_av, false};
        const uint32_t *cached = slot >= 0 ? cache + static_cast<int64_t>(slot) * row_words : nullptr;
        int nidx = nrows;
        bool fetched = false;   // the next row's description is in row .. row_seg
        int4 n_lo = make_int4(0, 0, 0, -1);   // the next row's description, in flight until the last slice
        longlong2 n_hi = make_longlong2(0, 0);
        // the current row is done with its description: the next row's replaces it
        auto take_next = [&]() {
            row = uniform(n_lo.x);
            a_lo = uniform(n_lo.y);
            a_hi = uniform(n_lo.z);
            slot = cache != nullptr ? uniform(n_lo.w) : -1;
            row_cb = POOL ? 0 : uniform(static_cast<int64_t>(n_hi.x));
            row_seg = POOL ? 0 : uniform(static_cast<int64_t>(n_hi.y));
        };

        // Pool output needs the row's entry count before its first write. A row of one region claims once that
        // region's count is known (below); a row spanning several regions counts its entries first, region by
        // region (a structure pass and a popcount each), and claims the total here.
        const bool multi_region = nwin > SH::REGION_WINS;
        if constexpr (POOL) {
            if (multi_region) {
                int total = 0;
                for (int rg0 = 0; rg0 < nwin; rg0 += SH::REGION_WINS) {
                    const int rg1 = nwin - rg0 < SH::REGION_WINS ? nwin : rg0 + SH::REGION_WINS;
                    const int64_t col0 = static_cast<int64_t>(rg0) * kRankWinCols;
                    const int ncw =
                        static_cast<int>(ncols - col0 < SH::REGION_COLS ? ncols - col0 : SH::REGION_COLS);
                    const int nwords = (ncw + 31) >> 5;
                    // the previous row's copy reads the bitmap words until every wave has left it
                    __syncthreads();
                    for (int i = threadIdx.x; i < RW; i += BLOCK) bw[i].x = 0u;
                    __syncthreads();
                    for_each_product_wg<BLOCK, V, false, true, true>(
                        M.a_col, M.a_val, a_lo, a_hi, BWindowRange{wtab, stride, rg0, rg1}, M.b_col, M.b_val, mark,
                        ctot, BitmapMark<2>{{}, &bw[0].x, static_cast<int>(col0)});
                    int cnt = 0;
                    for (int i = threadIdx.x; i < nwords; i += BLOCK) cnt += __popc(bw[i].x);
                    total += block_sum<BLOCK>(cnt, scratch);
                }
                if (threadIdx.x == 0) s_claim[0] = out.claim(row, total, &s_claim[1]);
                __syncthreads();
                cb = uniform(s_claim[0]);
                seg = uniform(s_claim[1]);
            }
        }
        int64_t done = 0;   // entries of the row emitted in earlier regions
        for (int rg0 = 0; rg0 < nwin; rg0 += SH::REGION_WINS) {
            const int rg1 = nwin - rg0 < SH::REGION_WINS ? nwin : rg0 + SH::REGION_WINS;
            const int64_t col0 = static_cast<int64_t>(rg0) * kRankWinCols;
            const int ncw = static_cast<int>(ncols - col0 < SH::REGION_COLS ? ncols - col0 : SH::REGION_COLS);
            const int nwords = (ncw + 31) >> 5;
            // 1. structure: the cached bitmap, or a structure pass (a region covering every column takes whole
            //    B rows, whose bounds come from B's row pointers rather than the larger window table). Either
            //    way the entry cache ends up holding each cached entry's column, value and part of B in the
            //    region.
            if (cached != nullptr) {
                int k = 0, lo = 0, hi = 0;
                double av = 0.0;
                const bool has_entry = ci < kCacheEntries && a_lo + ci < a_hi;
                if (rg0 == 0) {
                    // prefetched
                    k = pk;
                    av = to_d(pav);
                    lo = plo;
                    hi = phi;
                } else {
                    // later regions: the entries first (their loads then overlap the bitmap's), then the words
                    // this wave scans, all loaded before any is used
                    if (has_entry) k = e_col[ci];
                    const uint32_t *src = cached + static_cast<int64_t>(rg0) * WIN_WORDS;
#pragma unroll
                    for (int q = 0; q < WROWS; ++q) {
                        const int i = wbase + q * kWave + ln;
                        bits[q] = i < nwords ? __builtin_nontemporal_load(&src[i]) : 0u;
                    }
                    if (has_entry) {
                        const int32_t *t = wtab + static_cast<int64_t>(k) * stride;
                        lo = t[rg0];
                        hi = t[rg1];
                    }
                }
                if (ci < kCacheEntries) {
                    if (rg0 == 0) {
                        e_col[ci] = k;
                        e_av[ci] = av;
                    }
                    e_bs[ci] = lo;
                    e_len[ci] = hi - lo;
                    e_hi[ci] = hi;
                }
                ecache.col_ready = true;
                ecache.vals_ready = true;
            } else {
                // the previous slice's copy reads the bitmap words until every wave has left it
                __syncthreads();
                for (int i = threadIdx.x; i < RW; i += BLOCK) bw[i].x = 0u;
                __syncthreads();
                // (the .x words of bw, two words apart)
                const BitmapMark<2> mark_col{{}, &bw[0].x, static_cast<int>(col0)};
                if (nwin <= SH::REGION_WINS)
                    for_each_product_wg<BLOCK, V, false, true, true>(M.a_col, M.a_val, a_lo, a_hi,
                                                                     BRowRange{M.b_rp}, M.b_col, M.b_val, mark,
                                                                     ctot, mark_col, ecache);
                else
                    for_each_product_wg<BLOCK, V, false, true, true>(M.a_col, M.a_val, a_lo, a_hi,
                                                                     BWindowRange{wtab, stride, rg0, rg1}, M.b_col,
                                                                     M.b_val, mark, ctot, mark_col, ecache);
                ecache.col_ready = true;
                // the pass left each cached entry's region part in e_bs / e_len (written by this same thread)
                if (threadIdx.x < kCacheEntries) e_hi[threadIdx.x] = e_bs[threadIdx.x] + e_len[threadIdx.x];
#pragma unroll
                for (int q = 0; q < WROWS; ++q) bits[q] = bw[wbase + q * kWave + ln].x;
            }
            // 2. exclusive popcount prefix (lane-contiguous rows, so free of bank conflicts); each word is
            //    stored with its prefix. A 64-word row holds at most 2048 columns, so two rows' counts share
            //    one scan as the 16-bit halves of a word; the wave's total comes from the same scans.
            int region_total = 0;
            {
                static_assert(WROWS % 2 == 0 && kWave * 32 < 65536, "rows scanned in pairs of 16-bit counts");
                uint32_t cnt[WROWS];
                uint32_t inc2[WROWS / 2];
                int wtot = 0;
#pragma unroll
                for (int q = 0; q < WROWS; ++q) cnt[q] = __popc(bits[q]);
#pragma unroll
                for (int h = 0; h < WROWS / 2; ++h) {
                    inc2[h] = static_cast<uint32_t>(
                        wave_incl_sum(static_cast<int>(cnt[2 * h] | (cnt[2 * h + 1] << 16))));
                    const uint32_t t = __builtin_amdgcn_readlane(inc2[h], kWave - 1);
                    wtot += static_cast<int>((t & 0xffffu) + (t >> 16));
                }
                if (ln == 0) scratch[wv] = wtot;
                if (threadIdx.x == 0 && rg0 == 0) {
                    s_next = claimed;
                    claimed = atomicAdd(&ctrl->rank_next, 1);
                }
                __syncthreads();
                // one scan of the waves' totals gives this wave's first rank and the region's entry count
                const int wt = ln < NW ? scratch[ln] : 0;
                const int wincl = wave_incl_sum(wt);
                region_total = __builtin_amdgcn_readlane(wincl, NW - 1);
                int run = __builtin_amdgcn_readlane(wincl, wv) - __builtin_amdgcn_readlane(wt, wv);
#pragma unroll
                for (int h = 0; h < WROWS / 2; ++h) {
                    const uint32_t t = __builtin_amdgcn_readlane(inc2[h], kWave - 1);
                    const int lo = static_cast<int>(inc2[h] & 0xffffu), hi = static_cast<int>(inc2[h] >> 16);
                    bw[wbase + 2 * h * kWave + ln] =
                        make_uint2(bits[2 * h], static_cast<uint32_t>(run + lo - static_cast<int>(cnt[2 * h])));
                    run += static_cast<int>(t & 0xffffu);
                    bw[wbase + (2 * h + 1) * kWave + ln] = make_uint2(
                        bits[2 * h + 1], static_cast<uint32_t>(run + hi - static_cast<int>(cnt[2 * h + 1])));
                    run += static_cast<int>(t >> 16);
                }
            }
            if (rg0 == 0) {
                // the next row's description: in flight through this row's value passes
                nidx = uniform(s_next);
                if (nidx < nrows) {
                    const int z = opaque_zero();
                    const int4 *d = reinterpret_cast<const int4 *>(rr + nidx) + z;
                    n_lo = d[0];
                    n_hi = reinterpret_cast<const longlong2 *>(d)[1];
                }
            }
            if (POOL && !multi_region && threadIdx.x == 0) s_claim[0] = out.claim(row, region_total, &s_claim[1]);
            __syncthreads();
            if (POOL && !multi_region) {
                cb = uniform(s_claim[0]);
                seg = uniform(s_claim[1]);
            }
            // 3. rank slices: whole windows while they fit CAP entries; a window denser than CAP is taken in
            //    slices of CAP ranks. Lane jw holds the first rank of window jw (one LDS read for all windows).
            //    Window start ranks do not decrease, so the windows starting within CAP ranks of a slice's
            //    first rank are a prefix of the lanes: one ballot finds the slice's last window.
            const int nwr = rg1 - rg0;
            const int win_rank = ln <= nwr && ln * WIN_WORDS < nwords ? static_cast<int>(bw[ln * WIN_WORDS].y)
                                                                       : region_total;
            auto rank_at_window = [&](int jw) -> int { return __builtin_amdgcn_readlane(win_rank, jw); };
            int j = 0;
            int r0 = 0;              // first rank of the current slice
            int pj = 0, pj2 = nwr;   // windows of the slices the entry cache holds (first: the whole region)
            while (j < nwr) {
                const uint64_t fit = ballot(ln <= nwr && win_rank - r0 <= CAP);
                const int last_fit = 63 - static_cast<int>(__builtin_clzll(fit | 1ull));
                int j2 = last_fit < nwr ? last_fit : nwr;
                j2 = j2 > j + 1 ? j2 : j + 1;
                const int rend_w = rank_at_window(j2);
                const int r1 = rend_w - r0 > CAP ? r0 + CAP : rend_w;   // this slice covers ranks [r0, r1)
                // the row's last slice: the next row's loads go out while it is staged and copied
                const bool prefetch = rg1 == nwin && j2 == nwr && r1 == rend_w && nidx < nrows;
                // values
                const int lo_from = j == pj ? 0 : j == pj2 ? 1 : 2;
                const int hi_from = j2 == pj2 ? 0 : j2 == nwr ? 1 : 2;
                for_each_product_wg<BLOCK, V, true, true, false, OFF32>(
                    M.a_col, M.a_val, a_lo, a_hi,
                    SliceRange{wtab, stride, rg0 + j, rg0 + j2, lo_from, hi_from, e_bs, e_len, e_hi}, M.b_col,
                    M.b_val, mark, ctot, RankAccumulate{{}, bw, acc, static_cast<int>(col0), r0, r1}, ecache);
                ecache.vals_ready = true;
                pj = j;
                pj2 = j2;
                if (prefetch) {
                    take_next();
                    fetched = true;
                    if (slot >= 0) fetch_words(a_lo, a_hi, slot);
                }
                const int n = r1 - r0;
                // Emission of ranks [r0, r1). A slot's mark (the low half of its 8-byte accumulator slot for float
                // output, the stage array for double) is -1, or the index of the bitmap word holding that rank.
                if constexpr (SH::PACKED) {
                    // float output: round each accumulator once into the high half of its own slot; the low half
                    // becomes "no mark"
                    for (int i = threadIdx.x; i < n; i += BLOCK) {
                        const float v = static_cast<float>(acc[i]);
                        reinterpret_cast<uint2 *>(acc)[i] = make_uint2(0xffffffffu, __float_as_uint(v));
                    }
                    __syncthreads();
                }
                // Marks: every word holding ranks of the slice marks the first of them, and the one at a multiple
                // of 128 slots past r0 if it holds such a rank further on (a word holds at most 32 ranks, so at most
                // one). Each 128-slot block of the slice then starts on a mark.
                {
                    const int wa = j * WIN_WORDS;
                    const int wb = j2 * WIN_WORDS < nwords ? j2 * WIN_WORDS : nwords;
                    for (int wd = wa + static_cast<int>(threadIdx.x); wd < wb; wd += BLOCK) {
                        const uint2 e = bw[wd];
                        const int f = static_cast<int>(e.y) > r0 ? static_cast<int>(e.y) - r0 : 0;
                        const int l = static_cast<int>(e.y) + __popc(e.x) - r0;
                        const int le = l < n ? l : n;
                        if (f < le) {
                            rank_mark<SH::PACKED>(acc, stage, f, wd);
                            const int m128 = (f + 2 * kWave - 1) & ~(2 * kWave - 1);
                            if (m128 > f && m128 < le) rank_mark<SH::PACKED>(acc, stage, m128, wd);
                        }
                    }
                }
                __syncthreads();
                if (prefetch && slot >= 0) fetch_bounds(a_lo, a_hi);
                // copy the slice to C with coalesced stores, two slots per lane: wave w takes the 128-slot blocks
                // w, w + NW, ..., lane l slots 2l and 2l + 1 of the block. A slot's word is the last mark at or
                // before it in its block (a max-scan, since words increase with rank), its column the
                // (rank - word's first rank)-th set bit of that word. Marks and accumulators are cleared for the
                // next slice as they are read.
                {
                    int32_t *const colp = c_col + (cb + done + r0);   // uniform bases: 32-bit lane offsets
                    V *const valp = c_val + (cb + done + r0);
                    const int64_t lim = seg - (done + r0);   // slots at or past it are not written
                    // pairs of slots (even slot first) go out as one column store and one value store when both
                    // pairs are aligned to their size
                    const bool pair_aligned = (reinterpret_cast<uintptr_t>(colp) % (2 * sizeof(int32_t))) == 0 &&
                                              (reinterpret_cast<uintptr_t>(valp) % (2 * sizeof(V))) == 0;
                    for (int b0 = wv * 2 * kWave; b0 < n; b0 += 2 * BLOCK) {
                        const int i0 = b0 + 2 * ln;
                        int mk0 = -1, mk1 = -1;
                        V v0 = V(0), v1 = V(0);
                        if (i0 < n) {
                            // i0 is even: the two slots are one 16-byte read (and clear)
                            if constexpr (SH::PACKED) {
                                const uint4 u = reinterpret_cast<const uint4 *>(acc)[i0 >> 1];
                                mk0 = static_cast<int>(u.x);
                                v0 = static_cast<V>(__uint_as_float(u.y));
                                mk1 = static_cast<int>(u.z);
                                v1 = static_cast<V>(__uint_as_float(u.w));
                            } else {
                                const int2 m2 = reinterpret_cast<const int2 *>(stage)[i0 >> 1];
                                const double2 a2 = reinterpret_cast<const double2 *>(acc)[i0 >> 1];
                                reinterpret_cast<int2 *>(stage)[i0 >> 1] = make_int2(-1, -1);
                                mk0 = m2.x;
                                mk1 = m2.y;
                                v0 = static_cast<V>(a2.x);
                                v1 = static_cast<V>(a2.y);
                            }
                            reinterpret_cast<double2 *>(acc)[i0 >> 1] = make_double2(0.0, 0.0);
                        }
                        // slot i0 + 1's word: the last mark up to it; slot i0's: the last mark up to i0 - 1, or its own
                        const int w1 = wave_incl_max(mk1 > mk0 ? mk1 : mk0);
                        // (a DPP shift of the whole wave by one lane: lane 0 reads the identity)
                        const int w0 = max(__builtin_amdgcn_update_dpp(kMaxIdentity, w1, kDppWaveShr1, 0xf, 0xf, false), mk0);
                        if (i0 < n) {
                            const uint2 e0 = bw[w0];
                            const int p0 = select_set_bit(e0.x, r0 + i0 - static_cast<int>(e0.y));
                            const int c0 = static_cast<int>(col0) + w0 * 32 + p0;
                            // slot i0 + 1 holds the next set bit of the same word, or else the first rank of a
                            // later word, its lowest set bit (a mark at an odd slot is a word's first rank: marks
                            // inside a word sit at multiples of 128)
                            const uint32_t above = p0 < 31 ? e0.x >> (p0 + 1) : 0u;
                            int c1 = 0;
                            if (w1 == w0) {
                                c1 = c0 + 1 + static_cast<int>(__builtin_ctz(above | 0x80000000u));
                            } else {
                                const uint32_t x1 = bw[w1].x;
                                c1 = static_cast<int>(col0) + w1 * 32 + static_cast<int>(__builtin_ctz(x1 | 0x80000000u));
                            }
                            const bool two = i0 + 1 < n && i0 + 1 < lim;
                            if (pair_aligned && two) {
                                // streaming stores: C is written once, and must not push B out of the L2
                                store_pair_nt(colp + i0, c0, c1);
                                store_pair_nt(valp + i0, v0, v1);
                            } else {
                                if (i0 < lim) {
                                    __builtin_nontemporal_store(c0, &colp[i0]);
                                    __builtin_nontemporal_store(v0, &valp[i0]);
                                }
                                if (two) {
                                    __builtin_nontemporal_store(c1, &colp[i0 + 1]);
                                    __builtin_nontemporal_store(v1, &valp[i0 + 1]);
                                }
                            }
                        }
                    }
                }
                // no barrier here: the next accumulator and mark writes (the next slice's or row's value pass, then
                // its marks) come after the value pass's own barriers; the bitmap words the copy reads are rewritten
                // only after a barrier (the next region's or row's prefix, or the structure pass's clear); the entry
                // cache and the prefix scratch are not touched by the copy
                r0 = r1;
                if (r1 == rend_w) j = j2;   // the windows are done; otherwise the next slice of window j
            }
            done += region_total;
        }
        if (threadIdx.x == 0 && !POOL && done != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
        if (nidx >= nrows) break;
        if (!fetched) {
            // the last slice always prefetches; this keeps the loop right should it not
            take_next();
            if (slot >= 0) {
                fetch_words(a_lo, a_hi, slot);
                fetch_bounds(a_lo, a_hi);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Spill tier: persistent workgroups, each owning one slab of a bounded global
// pool (keys then doubles, slab_cap slots each). A launch takes the rows of one
// size class, with slabs sized for that class's largest table, so small rows
// run many workgroups at once and only the heaviest share few large slabs. A
// workgroup claims rows from the class's counter (the dynamic schedule:
// whoever finishes takes the next row), builds the row's hash table in its
// slab with global atomics, and in the numeric phase compacts the table into
// the row of C and merge-sorts it there, using the slab as the merge buffer.
// ---------------------------------------------------------------------------
constexpr int kSpillBlock = 512;
constexpr int kRunLen = 2048;      // LDS-sorted run length
constexpr int kMergeItems = 8;

template <typename V>
__device__ void merge_sort_segment(int32_t *__restrict__ col, V *__restrict__ val, int len,
                                   int32_t *__restrict__ tcol, V *__restrict__ tval,
                                   int32_t *s_keys, V *s_vals) {
    constexpr int BLOCK = kSpillBlock;
    // 1. sort runs of kRunLen in LDS
    for (int r0 = 0; r0 < len; r0 += kRunLen) {
        const int rl = (len - r0) < kRunLen ? (len - r0) : kRunLen;
        int n2 = 1;
        while (n2 < rl) n2 <<= 1;
        for (int i = threadIdx.x; i < n2; i += BLOCK) {
            if (i < rl) {
                s_keys[i] = col[r0 + i];
                s_vals[i] = val[r0 + i];
            } else {
                s_keys[i] = kPadKey;
            }
        }
        __syncthreads();
        for (int k = 2; k <= n2; k <<= 1) {
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int i = threadIdx.x; i < (n2 >> 1); i += BLOCK) {
                    const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));
                    const int hi = lo + j;
                    const bool up = (lo & k) == 0;
                    const int kl = s_keys[lo], kh = s_keys[hi];
                    if ((kl > kh) == up) {
                        s_keys[lo] = kh;
                        s_keys[hi] = kl;
                        const V t = s_vals[lo];
                        s_vals[lo] = s_vals[hi];
                        s_vals[hi] = t;
                    }
                }
                __syncthreads();
            }
        }
        for (int i = threadIdx.x; i < rl; i += BLOCK) {
            col[r0 + i] = s_keys[i];
            val[r0 + i] = s_vals[i];
        }
        __syncthreads();
    }
    // 2. merge runs pairwise, ping-ponging between the row and the slab
    int32_t *sc = col, *dc = tcol;
    V *sv = val, *dv = tval;
    for (int w = kRunLen; w < len; w <<= 1) {
        for (int p0 = 0; p0 < len; p0 += 2 * w) {
            const int lsz = (len - p0) < w ? (len - p0) : w;
            const int rsz = (len - p0 - lsz) < w ? (len - p0 - lsz) : w;
            const int total = lsz + rsz;
            const int32_t *L = sc + p0;
            const int32_t *R = L + lsz;
            for (int d0 = 0; d0 < total; d0 += BLOCK * kMergeItems) {
                const int d = d0 + static_cast<int>(threadIdx.x) * kMergeItems;
                if (d < total) {
                    int lo = d - rsz > 0 ? d - rsz : 0;
                    int hi = d < lsz ? d : lsz;
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (L[mid] < R[d - 1 - mid]) lo = mid + 1;
                        else hi = mid;
                    }
                    int i = lo, j = d - lo;
                    for (int t = 0; t < kMergeItems && d + t < total; ++t) {
                        const bool takeL = j >= rsz || (i < lsz && L[i] < R[j]);
                        if (takeL) {
                            dc[p0 + d + t] = L[i];
                            dv[p0 + d + t] = sv[p0 + i];
                            ++i;
                        } else {
                            dc[p0 + d + t] = R[j];
                            dv[p0 + d + t] = sv[p0 + lsz + j];
                            ++j;
                        }
                    }
                }
            }
        }
        __syncthreads();
        int32_t *tc = sc; sc = dc; dc = tc;
        V *tv = sv; sv = dv; dv = tv;
    }
    if (sc != col) {
        for (int i = threadIdx.x; i < len; i += BLOCK) {
            col[i] = sc[i];
            val[i] = sv[i];
        }
        __syncthreads();
    }
}

// One row of the spill tier, processed by the whole workgroup in its slab.
template <typename V, bool NUM>
__device__ __forceinline__ void spill_row(const Mats<V> &M, int row, const int64_t *__restrict__ pref,
                                          int64_t ncols, int32_t *__restrict__ keys, double *__restrict__ vals,
                                          int32_t *__restrict__ row_nnz, const RowSink &out,
                                          int32_t *__restrict__ c_col, V *__restrict__ c_val, Control *ctrl,
                                          int32_t *scratch, int32_t *s_keys, V *s_vals, int32_t *mark,
                                          int32_t *ctot, int64_t *s_claim) {
    constexpr int BLOCK = kSpillBlock;
    constexpr int NW = BLOCK / kWave;
    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    const int a_lo = M.a_rp[row], a_hi = M.a_rp[row + 1];
    int64_t bound;
    if (NUM && !out.pooled()) {
        bound = out.c_rp[row + 1] - out.c_rp[row];
    } else {
        const int64_t f = pref[a_hi] - pref[a_lo];
        bound = f < ncols ? f : ncols;
    }
    int log2t = ceil_log2(2 * (bound > 0 ? bound : 1));
    if (log2t < 6) log2t = 6;
    log2t = uniform(log2t);
    const int64_t T = int64_t(1) << log2t;   // the host guarantees T <= slab capacity
    for (int64_t i = threadIdx.x; i < T; i += BLOCK) {
        keys[i] = kEmptyKey;
        if (NUM) vals[i] = 0.0;
    }
    // make the cleared table visible at the device level before any atomic
    __threadfence();
    __syncthreads();

    int inserted = 0;
    bool overflow = false;
    for_each_product_wg<BLOCK, V, NUM>(
        M.a_col, M.a_val, a_lo, a_hi, BRowRange{M.b_rp}, M.b_col, M.b_val, mark, ctot,
        [&](int col, double prod) {
            uint32_t h = hash_slot(col, log2t);
            for (int64_t probe = 0; probe < T; ++probe) {
                const int old = atomicCAS(&keys[h], kEmptyKey, col);
                if (old == kEmptyKey || old == col) {
                    inserted += (old == kEmptyKey);
                    if (NUM) unsafeAtomicAdd(&vals[h], prod);
                    return;
                }
                h = (h + 1) & static_cast<uint32_t>(T - 1);
            }
            overflow = true;
        });
    if (overflow) atomicOr(&ctrl->error_flags, kErrProbeExhausted);
    if constexpr (!NUM) {
        const int total = block_sum<BLOCK>(inserted, scratch);
        if (threadIdx.x == 0) row_nnz[row] = total;
    } else {
        __threadfence();
        __syncthreads();
        // compact the table into the row of C (slot order), then sort it there
        int64_t cb, seg;
        if (!out.pooled()) {
            cb = out.c_rp[row];
            seg = out.c_rp[row + 1] - cb;
        } else {
            // the row's entries are its first insertions
            const int total = block_sum<BLOCK>(inserted, scratch);
            if (threadIdx.x == 0) s_claim[0] = out.claim(row, total, &s_claim[1]);
            __syncthreads();
            cb = uniform(s_claim[0]);
            seg = uniform(s_claim[1]);
        }
        int running = 0;
        for (int64_t s0 = 0; s0 < T; s0 += BLOCK) {
            const int64_t s = s0 + threadIdx.x;
            int k = kEmptyKey;
            double v = 0.0;
            if (s < T) {
                k = __hip_atomic_load(&keys[s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (k != kEmptyKey) v = __hip_atomic_load(&vals[s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            const int occ = k != kEmptyKey;
            int tot;
            const int ex = block_excl_scan<BLOCK>(occ, &tot, scratch);
            if (occ && running + ex < seg) {
                c_col[cb + running + ex] = k;
                c_val[cb + running + ex] = static_cast<V>(v);
            }
            running += tot;
        }
        if (threadIdx.x == 0 && !out.pooled() && running != seg) atomicOr(&ctrl->error_flags, kErrRowMismatch);
        __syncthreads();
        const int len = uniform(static_cast<int64_t>(running) < seg ? running : static_cast<int>(seg));
        merge_sort_segment<V>(c_col + cb, c_val + cb, len, keys, reinterpret_cast<V *>(vals), s_keys, s_vals);
    }
    __syncthreads();
}

template <typename V, bool NUM>
__global__ void __launch_bounds__(kSpillBlock) spill_kernel(
    Mats<V> M, const int32_t *__restrict__ rows, int32_t nrows, const int64_t *__restrict__ pref,
    int64_t ncols, char *__restrict__ pool, int64_t slab_cap, int32_t *__restrict__ row_nnz,
    RowSink out, int32_t *__restrict__ c_col, V *__restrict__ c_val,
    Control *ctrl, int32_t *next) {
    constexpr int NW = kSpillBlock / kWave;
    __shared__ int32_t s_row;
    __shared__ int64_t s_claim[2];   // pool output: the row's first entry and writable length
    __shared__ int32_t scratch[NW];
    __shared__ int32_t s_keys[NUM ? kRunLen : 1];
    __shared__ V s_vals[NUM ? kRunLen : 1];
    __shared__ int32_t marks[NW * kMarkInts];
    __shared__ int32_t ctot[kCtotInts];

    int32_t *keys = reinterpret_cast<int32_t *>(pool + static_cast<int64_t>(blockIdx.x) * slab_cap * 12);
    double *vals = reinterpret_cast<double *>(keys + slab_cap);
    int32_t *mark = marks + uniform(static_cast<int>(threadIdx.x) / kWave) * kMarkInts;
    init_marks(mark);

    // Rows are claimed one at a time from a shared counter until none are
    // left. The claimed index is read back into a scalar register so the loop
    // exit is uniform across the workgroup (every barrier below is reached by
    // all waves with all lanes active).
    for (;;) {
        if (threadIdx.x == 0) s_row = atomicAdd(next, 1);
        __syncthreads();
        const int ri = uniform(s_row);
        __syncthreads();
        if (ri >= nrows) break;
        spill_row<V, NUM>(M, rows[ri], pref, ncols, keys, vals, row_nnz, out, c_col, c_val, ctrl, scratch,
                          s_keys, s_vals, mark, ctot, s_claim);
    }
}

}  // namespace wsp
