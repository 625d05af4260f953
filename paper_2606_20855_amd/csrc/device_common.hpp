// Wave-level building blocks shared by the SpGEMM kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace wsp {

constexpr int kWave = 64;
constexpr int32_t kEmptyKey = -1;          // free hash slot
constexpr int32_t kPadKey = 0x7fffffff;    // sorts after every real column

// Control block bins. Rows are grouped by bin; each bin maps to one kernel
// shape. Dense and spill rows are split into classes by log2(products) with
// the heaviest class first, so launching a tier's bins in order hands out the
// longest rows first.
constexpr int kBinEmpty = 0;
constexpr int kBinTiny0 = 1;      // 1..4: segment widths 8, 16, 32, 64
constexpr int kNumTiny = 4;
constexpr int kBinHash0 = 5;      // 5..13: table sizes 2^6 .. 2^14
constexpr int kHashLog2Min = 6;
constexpr int kHashLog2Max = 14;
constexpr int kNumHash = kHashLog2Max - kHashLog2Min + 1;
constexpr int kNumClasses = 16;
constexpr int kBinDense0 = kBinHash0 + kNumHash;       // 14..29
constexpr int kBinSpill0 = kBinDense0 + kNumClasses;   // 30..45
constexpr int kNumBins = kBinSpill0 + kNumClasses;     // 46
constexpr int kMaxBins = 64;

enum : int32_t {
    kErrProbeExhausted = 1,   // a hash table filled up (structure larger than C.row_ptr says)
    kErrRowMismatch = 2,      // a row produced a different entry count than C.row_ptr
    kErrInvalidMatrix = 4,    // validation found a non-canonical input
};

// Record of what the last symbolic phase left in the workspace for the
// numeric phase: the column sets (bitmaps) of dense rows. It names the inputs
// and the layout it was made for and a checksum of C.row_ptr; the numeric
// phase uses the bitmaps only if all of them match its own call. magic is 0
// while a symbolic phase is running or after it failed.
struct Stamp {
    uint64_t magic;
    uint64_t a_rp, a_col, b_rp, b_col;
    int64_t a_nrows, a_ncols, a_nnz, b_nrows, b_ncols, b_nnz;
    int64_t off_slot, off_cache, row_words, cache_rows;
    int64_t cached_rows;   // rows that received a cache slot
    uint64_t rp_sum;
    // The numeric phase's binning of the rows by C's exact row counts, done once C.row_ptr was known, with
    // these settings (num_bins 1), and B's window table (wtab 1): the numeric phase takes them when its own
    // settings are the same.
    int64_t num_bins, wtab;
    int64_t nb_dense_min_nnz;
    int32_t nb_tiny_max, nb_hash_log2_max, nb_force_spill, nb_dense_ok;
};
constexpr uint64_t kStampMagic = 0x57535f5354525543ull;

// Device-side control block, zeroed at the start of each phase and copied to
// the host once the rows have been binned.
struct Control {
    int64_t total_products;
    int64_t spill_max_bound;
    int64_t c_nnz;
    unsigned long long pool_claimed;   // single pass: pool entries the rows have claimed
    int32_t spill_next[kNumClasses];   // the spill tier's row claims, one counter per size class
    int32_t error_flags;
    int32_t has_zero_values;   // some A or B value could give a zero product
    int32_t rank_next;         // the rank kernel's row claims
    uint64_t rp_sum;           // numeric: checksum of the C.row_ptr it was given
    int32_t bin_count[kMaxBins];
    int32_t bin_offset[kMaxBins];
    int32_t bin_cursor[kMaxBins];
    int64_t stat_products[kMaxBins];
    int64_t stat_annz[kMaxBins];
    int64_t stat_cnnz[kMaxBins];
};

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Where a numeric kernel writes the rows of C. Without a claim counter the
// rows go to plain CSR at C.row_ptr, which the symbolic phase computed. With
// one (the single pass, with sharded output) a row's entry count is known only
// once the row is computed: the row then claims that many entries of the pool
// from the shared counter (the first and only writer of a row claims its
// storage), records where in row_off / row_nnz, and is written there. A row
// that would pass the pool's capacity writes nothing, but the counter still
// grows, so it ends at the entry count of C.
struct RowSink {
    const int64_t *c_rp = nullptr;
    unsigned long long *claimed = nullptr;
    int64_t *row_off = nullptr;
    int32_t *row_nnz = nullptr;
    int64_t cap = 0;
    __device__ __forceinline__ bool pooled() const { return claimed != nullptr; }
    // Pool output: claims `count` entries for `row` and returns the first. *len
    // is how many the row may write: count, or 0 when the pool is too small.
    __device__ __forceinline__ int64_t claim(int row, int count, int64_t *len) const {
        const int64_t off = static_cast<int64_t>(atomicAdd(claimed, static_cast<unsigned long long>(count)));
        row_off[row] = off;
        row_nnz[row] = count;
        *len = off + count <= cap ? count : 0;
        return off;
    }
};

// 64-bit value of lane `src` of each group of `width` lanes.
__device__ __forceinline__ int64_t shfl_i64(int64_t x, int src, int width) {
    const int lo = __shfl(static_cast<int>(x), src, width);
    const int hi = __shfl(static_cast<int>(x >> 32), src, width);
    return static_cast<int64_t>((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}

// Lane mask of a condition (bit l set where lane l's condition holds),
// straight from the compare's scalar mask.
__device__ __forceinline__ uint64_t ballot(bool b) { return __builtin_amdgcn_ballot_w64(b); }

// Values every lane of the workgroup holds identically (read back from LDS
// after a barrier) are moved to scalar registers, so loops and branches that
// depend on them compile as uniform control flow. Barriers then never sit in
// a region the compiler treats as divergent.
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int64_t uniform(int64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(x) >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ __forceinline__ double to_d(float x) { return static_cast<double>(x); }
__device__ __forceinline__ double to_d(double x) { return x; }

// Inclusive prefix sum within aligned groups of W lanes (W a power of two).
template <int W>
__device__ __forceinline__ int group_incl_scan(int x) {
    const int gl = lane_id() & (W - 1);
#pragma unroll
    for (int o = 1; o < W; o <<= 1) {
        const int y = __shfl_up(x, o, W);
        if (gl >= o) x += y;
    }
    return x;
}

// Within a group of W lanes holding a non-decreasing `incl`, the number of
// lanes whose value is <= q. With incl the inclusive prefix of per-lane
// lengths and q < incl[W-1], this is the lane that owns element q.
template <int W>
__device__ __forceinline__ int group_count_le(int incl, int q) {
    int c = 0;
#pragma unroll
    for (int step = W / 2; step >= 1; step >>= 1) {
        const int v = __shfl(incl, c + step - 1, W);
        if (v <= q) c += step;
    }
    return c;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

// Block-wide sum; every thread gets the result. `scratch` holds BLOCK/64 T.
template <int BLOCK, typename T>
__device__ __forceinline__ T block_sum(T x, T *scratch) {
    constexpr int NW = BLOCK / kWave;
    x = wave_sum(x);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) scratch[w] = x;
    __syncthreads();
    T t = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) t += scratch[i];
    __syncthreads();
    return uniform(t);
}

// Block-wide exclusive prefix sum of int; returns the exclusive value and the
// block total. `scratch` holds BLOCK/64 ints.
template <int BLOCK>
__device__ __forceinline__ int block_excl_scan(int x, int *total, int *scratch) {
    constexpr int NW = BLOCK / kWave;
    const int incl = group_incl_scan<kWave>(x);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) scratch[w] = incl;
    __syncthreads();
    int before = 0, t = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const int s = scratch[i];
        before += (i < w) ? s : 0;
        t += s;
    }
    __syncthreads();
    *total = uniform(t);
    return before + incl - x;
}

// Multiplicative (Fibonacci) hashing: the top `log2t` bits of key * 2^32/phi.
__device__ __forceinline__ uint32_t hash_slot(int32_t key, int log2t) {
    return (static_cast<uint32_t>(key) * 2654435761u) >> (32 - log2t);
}

__host__ __device__ __forceinline__ int ceil_log2(int64_t x) {
    int l = 0;
    while ((int64_t(1) << l) < x) ++l;
    return l;
}

// ---------------------------------------------------------------------------
// Wave-wide inclusive scans with DPP lane moves (row shifts within 16-lane
// rows, then row broadcasts of lanes 15 and 31): VALU only, no LDS traffic.
// ---------------------------------------------------------------------------
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;
constexpr int kDppWaveShr1 = 0x138;   // whole-wave shift right by one lane

__device__ __forceinline__ int wave_incl_sum(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr1, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr2, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr4, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr8, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast15, 0xa, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast31, 0xc, 0xf, false);
    return v;
}

// Inclusive max-scan. Lanes a DPP step does not feed read INT_MIN, the identity
// of signed max, which lets the compiler fuse each step into one max with a DPP
// operand.
constexpr int kMaxIdentity = static_cast<int>(0x80000000u);
__device__ __forceinline__ int wave_incl_max(int v) {
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowShr1, 0xf, 0xf, false), v);
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowShr2, 0xf, 0xf, false), v);
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowShr4, 0xf, 0xf, false), v);
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowShr8, 0xf, 0xf, false), v);
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowBcast15, 0xa, 0xf, false), v);
    v = max(__builtin_amdgcn_update_dpp(kMaxIdentity, v, kDppRowBcast31, 0xc, 0xf, false), v);
    return v;
}

// Orders a wave's LDS accesses to different addresses (compiler and hardware).
__device__ __forceinline__ void wave_lds_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

// Per-wave LDS scratch of kMarkInts ints used by for_each_product_wg to
// locate the A entries of blocks that span several of them. It must hold -1
// everywhere before the first call; for_each_product_wg leaves it that way.
constexpr int kScalarOwners = 4;      // entries per block resolved with scalar reads (4 measured best of 4, 8, 16)
constexpr int kMarkInts = 2 * kWave;   // short-row iteration: marks of two blocks at once
constexpr int kMarkIntsLong = kWave;   // long-row iteration: one block at a time

// Sets this wave's mark array (n ints) to -1.
__device__ __forceinline__ void init_marks(int32_t *mark, int n = kMarkInts) {
    for (int i = lane_id(); i < n; i += kWave) mark[i] = -1;
    wave_lds_fence();
}

__device__ __forceinline__ double readlane_d(double x, int lane) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(x), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(x), lane);
    return __hiloint2double(hi, lo);
}

// A visitor deriving from TwoPhaseVisit splits a visit into k = pre(col), a
// lookup, and post(k, prod), the update; operator()(col, prod) must equal
// post(pre(col), prod), and post(-1, prod) must do nothing. safe_col() is a
// column pre() accepts whatever the visit. Steps then issue all lookups before
// any update, and dead lanes look up safe_col() (no branch around a lookup).
struct TwoPhaseVisit {};

// quad permutations: every lane of a pair (2i, 2i + 1) reads lane 2i, or lane 2i + 1
constexpr int kDppPairEven = 0xA0;   // quad_perm [0, 0, 2, 2]
constexpr int kDppPairOdd = 0xF5;    // quad_perm [1, 1, 3, 3]

// Marks columns in an LDS bitmap whose word j is bm[j * STRIDE], columns taken
// relative to col0. Several lanes of one atomic instruction that hit the same
// word are serialised by LDS, and the lanes of a block over a long B slice
// hold increasing columns, so neighbours often share a word. Lanes therefore
// work in pairs (2i, 2i + 1): the odd lane also sets the even lane's bit when
// both name the same word, and the even lane issues its atomic only when they
// do not. Every bit is set whatever the order of the columns. The pair
// exchange is a quad permutation, so the whole wave must be active (the block
// steps of for_each_product_wg are). A dead lane's post gets -1 and marks
// nothing; its word (-1) matches no live lane's.
template <int STRIDE>
struct BitmapMark : TwoPhaseVisit {
    uint32_t *bm;
    int col0;
    __device__ __forceinline__ int pre(int col) const { return col - col0; }
    __device__ __forceinline__ int safe_col() const { return col0; }
    __device__ __forceinline__ void post(int rel, double) const {
        const int w = rel >> 5;   // -1 for a dead lane
        const int bit = static_cast<int>(1u << (rel & 31));
        const int w_even = __builtin_amdgcn_mov_dpp(w, kDppPairEven, 0xf, 0xf, false);
        const int bit_even = __builtin_amdgcn_mov_dpp(bit, kDppPairEven, 0xf, 0xf, false);
        const int w_odd = __builtin_amdgcn_mov_dpp(w, kDppPairOdd, 0xf, 0xf, false);
        if (rel >= 0 && ((lane_id() & 1) || w_odd != w))
            atomicOr(&bm[w * STRIDE], static_cast<uint32_t>(w_even == w ? (bit | bit_even) : bit));
    }
    __device__ __forceinline__ void operator()(int col, double prod) const { post(pre(col), prod); }
    // Four consecutive columns of one B slice, in one lane (a span step of entry-aligned blocks, see
    // chunk_blocks_aligned): each run of columns in one word ORs its bits into the run's last column, which
    // alone issues the atomic. As above, any column order gives the same bitmap.
    __device__ __forceinline__ void run4(int c0, int c1, int c2, int c3) const {
        const int r0 = c0 - col0, r1 = c1 - col0, r2 = c2 - col0, r3 = c3 - col0;
        const int w0 = r0 >> 5, w1 = r1 >> 5, w2 = r2 >> 5, w3 = r3 >> 5;
        const uint32_t b0 = 1u << (r0 & 31), b1 = 1u << (r1 & 31), b2 = 1u << (r2 & 31), b3 = 1u << (r3 & 31);
        const bool s01 = w0 == w1, s12 = w1 == w2, s23 = w2 == w3;
        const uint32_t p1 = b1 | (s01 ? b0 : 0u);
        const uint32_t p2 = b2 | (s12 ? p1 : 0u);
        const uint32_t p3 = b3 | (s23 ? p2 : 0u);
        if (!s01) atomicOr(&bm[w0 * STRIDE], b0);
        if (!s12) atomicOr(&bm[w1 * STRIDE], p1);
        if (!s23) atomicOr(&bm[w2 * STRIDE], p2);
        atomicOr(&bm[w3 * STRIDE], p3);
    }
};
// Whether a visitor takes four consecutive columns of one lane at once (run4).
template <typename T, typename = void>
struct has_run4 : std::false_type {};
template <typename T>
struct has_run4<T, std::void_t<decltype(std::declval<const T &>().run4(0, 0, 0, 0))>> : std::true_type {};

// Processes blocks [lb0, lb1) (block = 64 consecutive products) of one
// 64-entry A chunk whose lanes hold (boff, av, len, incl): the shared body of
// the product iterators. `mark` is this wave's LDS mark array (all -1).
//
// Long B slices (the bulk of the products on skewed inputs) take a span
// step: kSpanBlocks blocks that all lie inside one entry are read with one
// address computation (lane l takes products l, l+64, l+128, l+192) and
// visited without any per-product branch. Other blocks go U at a time in a
// general step (U = 4 for long rows, 2 for short ones). Within a step every
// lane loads (a dead lane from entry 0, which exists whenever a block does),
// so the step's loads are issued back to back and waited for once.
constexpr int kSpanBlocks = 4;

// base[ix] for ix >= 0. With OFF32 the element's byte offset is formed in 32
// bits (one shift, and the load takes the base from scalar registers), which
// the caller may ask for only when every offset it uses is below 2^32.
template <bool OFF32, typename T>
__device__ __forceinline__ T load_at(const T *__restrict__ base, int ix) {
    if constexpr (OFF32)
        return *reinterpret_cast<const T *>(reinterpret_cast<const char *>(base) +
                                            static_cast<uint32_t>(ix) * static_cast<uint32_t>(sizeof(T)));
    else
        return base[ix];
}

template <typename V, bool VALUES, bool LONG, bool OFF32, typename Visit>
__device__ __forceinline__ void chunk_blocks(int boff, double av, int len, int incl, int tot, int lb0, int lb1,
                                             const int32_t *__restrict__ b_col, const V *__restrict__ b_val,
                                             int32_t *mark, Visit &visit) {
    constexpr int U = LONG ? 4 : 2;
    constexpr int SB = kSpanBlocks;
    const int ln = lane_id();
    const int excl = incl - len;
    // first product of the lane's entry, or INT_MAX for an entry without products: "an entry with products
    // starts at or before q" is then one compare
    const int start = len > 0 ? excl : 0x7fffffff;
    // the span step from block lb: returns false (doing nothing) when blocks lb .. lb + SB - 1 are not all
    // inside one entry's slice
    auto span_step = [&](int lb) -> bool {
        constexpr int NB = SB;
        const int base = lb * kWave;
        const uint64_t before = ballot(start <= base);
        const int o = 63 - __clzll(before | 1ull);
        // the entry's products reach past the span's last one (so the span is also below tot)
        if (__builtin_amdgcn_readlane(incl, o) <= base + NB * kWave - 1) return false;
        const int64_t b0 = static_cast<int64_t>(__builtin_amdgcn_readlane(boff, o)) + base;
        const int32_t *cp = b_col + b0 + ln;
        const V *vp = b_val + b0 + ln;
        const double a = VALUES ? readlane_d(av, o) : 0.0;
        int c[NB];
        V v[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            c[u] = cp[u * kWave];
            if (VALUES) v[u] = vp[u * kWave];
        }
        // keep the compiler from sinking a load into its use
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            asm volatile("" : "+v"(c[u]));
            if (VALUES) asm volatile("" : "+v"(v[u]));
        }
        if constexpr (std::is_base_of<TwoPhaseVisit, Visit>::value) {
            int k[NB];
#pragma unroll
            for (int u = 0; u < NB; ++u) k[u] = visit.pre(c[u]);
#pragma unroll
            for (int u = 0; u < NB; ++u) visit.post(k[u], VALUES ? a * to_d(v[u]) : 0.0);
        } else {
#pragma unroll
            for (int u = 0; u < NB; ++u) visit(c[u], VALUES ? a * to_d(v[u]) : 0.0);
        }
        return true;
    };
    for (int lb = lb0; lb < lb1;) {
        if (lb + SB <= lb1 && span_step(lb)) {
            lb += SB;
            continue;
        }
        // general step: U blocks
        int ix[U];
        double aval[U];
        bool live[U];
        if constexpr (LONG) {
            // Each block resolved on its own. A block inside one entry takes
            // that entry's data from scalar registers; a block spanning up to
            // kScalarOwners entries assigns them to lanes with scalar reads of
            // each entry's data (no LDS round trip); only blocks spanning more
            // entries use the LDS marks and a max-scan.
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int base = (lb + u) * kWave;
                const int p = base + ln;
                live[u] = lb + u < lb1 && p < tot;
                ix[u] = 0;
                aval[u] = 0.0;
                if (lb + u >= lb1) continue;
                const uint64_t bf = ballot(start <= base);
                const int ob = 63 - __clzll(bf | 1ull);
                const int last = (base + kWave < tot ? base + kWave : tot) - 1;
                const uint64_t bl = ballot(start <= last);
                const int oe = 63 - __clzll(bl | 1ull);
                if (oe - ob < kScalarOwners) {
                    int bo = __builtin_amdgcn_readlane(boff, ob);
                    double a = VALUES ? readlane_d(av, ob) : 0.0;
                    for (int e = ob + 1; e <= oe; ++e) {
                        const int e_start = __builtin_amdgcn_readlane(start, e);
                        const int e_boff = __builtin_amdgcn_readlane(boff, e);
                        const double e_av = VALUES ? readlane_d(av, e) : 0.0;
                        if (p >= e_start) {
                            bo = e_boff;
                            a = e_av;
                        }
                    }
                    ix[u] = bo + p;
                    aval[u] = a;
                } else {
                    if (len > 0 && excl > base && excl < base + kWave) mark[excl - base] = ln;
                    wave_lds_fence();
                    int m = mark[ln];
                    mark[ln] = -1;
                    m = wave_incl_max(m);
                    const int o = m > ob ? m : ob;
                    wave_lds_fence();
                    ix[u] = __shfl(boff, o, kWave) + p;
                    aval[u] = VALUES ? __shfl(av, o, kWave) : 0.0;
                }
                if (!live[u]) ix[u] = 0;
            }
        } else {
            // Short slices: if every block lies inside one entry, the entries'
            // data come from scalar registers; otherwise all U blocks share one
            // LDS mark/max-scan round.
            int ob[U];
            bool fast = true;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int base = (lb + u) * kWave;
                const uint64_t before = ballot(start <= base);
                ob[u] = 63 - __clzll(before | 1ull);
                const int last = (base + kWave < tot ? base + kWave : tot) - 1;
                fast = fast && (lb + u >= lb1 || __builtin_amdgcn_readlane(incl, ob[u]) > last);
            }
            int bidx[U];
            if (fast) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    bidx[u] = __builtin_amdgcn_readlane(boff, ob[u]) + (lb + u) * kWave + ln;
                    aval[u] = VALUES ? readlane_d(av, ob[u]) : 0.0;
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int base = (lb + u) * kWave;
                    if (len > 0 && excl > base && excl < base + kWave) mark[u * kWave + excl - base] = ln;
                }
                wave_lds_fence();
                int o[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    int m = mark[u * kWave + ln];
                    mark[u * kWave + ln] = -1;
                    m = wave_incl_max(m);
                    o[u] = m > ob[u] ? m : ob[u];
                }
                wave_lds_fence();
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    bidx[u] = __shfl(boff, o[u], kWave) + (lb + u) * kWave + ln;
                    aval[u] = VALUES ? __shfl(av, o[u], kWave) : 0.0;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                live[u] = lb + u < lb1 && (lb + u) * kWave + ln < tot;
                ix[u] = live[u] ? bidx[u] : 0;
            }
        }
        int craw[U];
        V vraw[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            craw[u] = load_at<OFF32>(b_col, ix[u]);
            if (VALUES) vraw[u] = load_at<OFF32>(b_val, ix[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            asm volatile("" : "+v"(craw[u]));
            if (VALUES) asm volatile("" : "+v"(vraw[u]));
        }
        if constexpr (std::is_base_of<TwoPhaseVisit, Visit>::value) {
            int k[U];
#pragma unroll
            for (int u = 0; u < U; ++u) k[u] = visit.pre(live[u] ? craw[u] : visit.safe_col());
#pragma unroll
            for (int u = 0; u < U; ++u) visit.post(live[u] ? k[u] : -1, VALUES ? aval[u] * to_d(vraw[u]) : 0.0);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (live[u]) visit(craw[u], VALUES ? aval[u] * to_d(vraw[u]) : 0.0);
            }
        }
        lb += U;
    }
}

// LDS copy of the first kCacheEntries A entries of a row, filled by step 1 of
// a for_each_product_wg call (its slices in the call's range, its value) and
// read back when step 3 loads a chunk, so a chunk costs an LDS read instead of
// two dependent global round trips. `col` (the entries' columns) stays valid
// for later calls on the same row once `col_ready` is set, which saves those
// calls one round trip in step 1 too. A null `col` disables the cache.
constexpr int kCacheChunks = 4;
constexpr int kCacheEntries = kCacheChunks * kWave;
// Long rows: blocks aligned to entries. Entry e of a 64-entry chunk (lane e)
// owns the ceil(len_e / 64) consecutive blocks from bstart_e, block k of the
// entry taking products 64k .. 64k+63 of its slice (an entry's last block may
// be partial). Every block thus has exactly one entry, found with one ballot,
// and a step of kSpanBlocks full blocks of one entry is read with one address
// computation. Processes blocks [lb0, lb1) of the chunk whose lanes hold
// (bs, av, len, bstart, nblk). As in chunk_blocks every lane of a step loads
// (a dead lane from its block's own entry), so the loads go out back to back.
template <typename V, bool VALUES, typename Visit>
__device__ __forceinline__ void chunk_blocks_aligned(int bs, double av, int len, int bstart, int nblk, int lb0,
                                                     int lb1, const int32_t *__restrict__ b_col,
                                                     const V *__restrict__ b_val, Visit &visit) {
    constexpr int SB = kSpanBlocks;
    const int ln = lane_id();
    // first block of the lane's entry, or INT_MAX for an entry without products
    const int bfirst = nblk > 0 ? bstart : 0x7fffffff;
    for (int lb = lb0; lb < lb1;) {
        const uint64_t m0 = ballot(bfirst <= lb);
        const int o = 63 - __clzll(m0 | 1ull);
        const int k = lb - __builtin_amdgcn_readlane(bstart, o);   // block of entry o
        const int len_o = __builtin_amdgcn_readlane(len, o);
        if (lb + SB <= lb1 && (k + SB) * kWave <= len_o) {
            // every span step of entry o inside [lb, lb1), its data read from the lanes once
            int nsp = (len_o / kWave - k) / SB;
            const int nmax = (lb1 - lb) / SB;
            nsp = nsp < nmax ? nsp : nmax;
            const int64_t bo = static_cast<int64_t>(__builtin_amdgcn_readlane(bs, o)) + k * kWave;
            const double a = VALUES ? readlane_d(av, o) : 0.0;
            if constexpr (!VALUES && has_run4<Visit>::value) {
                // structure only: lane l takes products 4l .. 4l + 3 of each span with one 16-byte load (4-byte
                // aligned), so a lane's columns sharing a word are merged in registers before any LDS atomic;
                // four spans' loads go out before the first is visited
                static_assert(SB == 4, "four consecutive columns per lane");
                typedef int32_t i32x4u __attribute__((ext_vector_type(4), aligned(4)));
                const int32_t *qp = b_col + bo + 4 * ln;
                int t = 0;
                for (; t + 3 < nsp; t += 4) {
                    i32x4u q0 = *reinterpret_cast<const i32x4u *>(qp + t * (SB * kWave));
                    i32x4u q1 = *reinterpret_cast<const i32x4u *>(qp + (t + 1) * (SB * kWave));
                    i32x4u q2 = *reinterpret_cast<const i32x4u *>(qp + (t + 2) * (SB * kWave));
                    i32x4u q3 = *reinterpret_cast<const i32x4u *>(qp + (t + 3) * (SB * kWave));
                    asm volatile("" : "+v"(q0));
                    asm volatile("" : "+v"(q1));
                    asm volatile("" : "+v"(q2));
                    asm volatile("" : "+v"(q3));
                    visit.run4(q0.x, q0.y, q0.z, q0.w);
                    visit.run4(q1.x, q1.y, q1.z, q1.w);
                    visit.run4(q2.x, q2.y, q2.z, q2.w);
                    visit.run4(q3.x, q3.y, q3.z, q3.w);
                }
                for (; t < nsp; ++t) {
                    const i32x4u q = *reinterpret_cast<const i32x4u *>(qp + t * (SB * kWave));
                    visit.run4(q.x, q.y, q.z, q.w);
                }
                lb += nsp * SB;
                continue;
            }
            for (int t = 0; t < nsp; ++t) {
                const int64_t b0 = bo + t * (SB * kWave);
                const int32_t *cp = b_col + b0 + ln;
                const V *vp = b_val + b0 + ln;
                int c[SB];
                V v[SB];
#pragma unroll
                for (int u = 0; u < SB; ++u) {
                    c[u] = cp[u * kWave];
                    if (VALUES) v[u] = vp[u * kWave];
                }
                // keep the compiler from sinking a load into its use
#pragma unroll
                for (int u = 0; u < SB; ++u) {
                    asm volatile("" : "+v"(c[u]));
                    if (VALUES) asm volatile("" : "+v"(v[u]));
                }
                if constexpr (std::is_base_of<TwoPhaseVisit, Visit>::value) {
                    int kk[SB];
#pragma unroll
                    for (int u = 0; u < SB; ++u) kk[u] = visit.pre(c[u]);
#pragma unroll
                    for (int u = 0; u < SB; ++u) visit.post(kk[u], VALUES ? a * to_d(v[u]) : 0.0);
                } else {
#pragma unroll
                    for (int u = 0; u < SB; ++u) visit(c[u], VALUES ? a * to_d(v[u]) : 0.0);
                }
            }
            lb += nsp * SB;
            continue;
        }
        // SB blocks, each inside one entry
        int ix[SB];
        double aval[SB];
        bool live[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int b = lb + u;
            live[u] = false;
            ix[u] = 0;
            aval[u] = 0.0;
            if (b < lb1) {
                const uint64_t m = ballot(bfirst <= b);
                const int e = 63 - __clzll(m | 1ull);
                const int p = (b - __builtin_amdgcn_readlane(bstart, e)) * kWave + ln;
                live[u] = p < __builtin_amdgcn_readlane(len, e);
                ix[u] = __builtin_amdgcn_readlane(bs, e) + (live[u] ? p : 0);
                aval[u] = VALUES ? readlane_d(av, e) : 0.0;
            }
        }
        int craw[SB];
        V vraw[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            craw[u] = b_col[ix[u]];
            if (VALUES) vraw[u] = b_val[ix[u]];
        }
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            asm volatile("" : "+v"(craw[u]));
            if (VALUES) asm volatile("" : "+v"(vraw[u]));
        }
        if constexpr (std::is_base_of<TwoPhaseVisit, Visit>::value) {
            int kk[SB];
#pragma unroll
            for (int u = 0; u < SB; ++u) kk[u] = visit.pre(live[u] ? craw[u] : visit.safe_col());
#pragma unroll
            for (int u = 0; u < SB; ++u) visit.post(live[u] ? kk[u] : -1, VALUES ? aval[u] * to_d(vraw[u]) : 0.0);
        } else {
#pragma unroll
            for (int u = 0; u < SB; ++u) {
                if (live[u]) visit(craw[u], VALUES ? aval[u] * to_d(vraw[u]) : 0.0);
            }
        }
        lb += SB;
    }
}

struct EntryCache {
    int32_t *col = nullptr;
    int32_t *bs = nullptr;
    int32_t *len = nullptr;
    double *av = nullptr;
    bool col_ready = false;    // col holds the entries' columns
    bool vals_ready = false;   // av holds the entries' values
};

// A range functor with a member cached(k, ci) gives the slices of entries held
// in the entry cache from there (ci: the entry's cache index) instead of from
// memory.
template <typename R, typename = void>
struct has_cached_bounds : std::false_type {};
template <typename R>
struct has_cached_bounds<R, std::void_t<decltype(std::declval<const R &>().cached(0, 0))>> : std::true_type {};

// Visits every product a * b of A entries [a_lo, a_hi) of one row: visit(col,
// prod) with col = B.col_idx[b] and prod = A.val[a] * B.val[b] formed in double
// (0 when VALUES is false). `range(k)` gives the slice [x, y) of B's entry
// arrays that multiplies A entry k (a whole row of B, or its part inside
// column windows).
//
// Products are flattened per 64-entry chunk of A: lane l of a chunk holds the
// prefix sum of slice lengths, and block t of the chunk covers products
// 64t .. 64t+63, lane j of the block taking product 64t + j. Consecutive lanes
// therefore read consecutive B entries whenever a slice is long, and no lane
// idles on short slices. Entries are taken in groups of up to kMaxChunks
// chunks of 64. For each group:
//   1. wave w measures chunks w, w+NW, ...: its count of 64-product blocks;
//   2. one wave scans the counts into block offsets (ctot, in LDS);
//   3. the blocks are shared out. For short rows (LONG false) wave w takes
//      the contiguous range [w*nb/NW, (w+1)*nb/NW). For long rows waves claim
//      runs of consecutive blocks from an LDS counter until none are left: a
//      block costs more where slices are short (entry boundaries inside
//      blocks) than inside a long slice, so claiming keeps the waves finishing
//      together (on short rows the claims would cost more than they save).
//      Either way a wave moves forward through the chunks, keeping its current
//      one in registers.
// LONG also selects the general-step shape (see chunk_blocks). ALIGNED (for
// visits over whole B rows, where slices are long) replaces the flattening by
// entry-aligned blocks (see chunk_blocks_aligned): more blocks, but never a
// block shared by two entries. OFF32 (see load_at) forms the general steps' B
// offsets in 32 bits: only for B with nnz * sizeof(V) <= 2^32.
// All threads of the workgroup must call it. ctot holds kCtotInts ints of LDS.
constexpr int kMaxChunks = 256;
constexpr int kCtotInts = kMaxChunks + 2;   // block offsets, total, claim counter
constexpr int kUnitBlocks = 4;

template <int BLOCK, typename V, bool VALUES, bool LONG = false, bool ALIGNED = false, bool OFF32 = false,
          typename RangeF, typename Visit>
__device__ __forceinline__ void for_each_product_wg(const int32_t *__restrict__ a_col,
                                                    const V *__restrict__ a_val, int a_lo, int a_hi,
                                                    RangeF range, const int32_t *__restrict__ b_col,
                                                    const V *__restrict__ b_val, int32_t *mark, int32_t *ctot,
                                                    Visit visit, EntryCache cache = EntryCache{}) {
    constexpr int NW = BLOCK / kWave;
    const int wv = uniform(static_cast<int>(threadIdx.x) / kWave);
    const int ln = lane_id();
    int32_t *claim = ctot + kMaxChunks + 1;
    for (int g0 = a_lo; g0 < a_hi; g0 += kMaxChunks * kWave) {
        const int g1 = (a_hi - g0) < kMaxChunks * kWave ? a_hi : g0 + kMaxChunks * kWave;
        const int nch = (g1 - g0 + kWave - 1) / kWave;
        const bool use_cache = cache.col != nullptr && g0 == a_lo;
        // 1. blocks per chunk
        for (int c = wv; c < nch; c += NW) {
            const int a = g0 + c * kWave + ln;
            const bool cached = use_cache && c < kCacheChunks;
            const int ci = c * kWave + ln;
            int len = 0;
            if (a < g1) {
                int k;
                if (cached && cache.col_ready) k = cache.col[ci];
                else k = a_col[a];
                double av = 0.0;
                if (VALUES && cached && !cache.vals_ready) av = to_d(a_val[a]);
                int2 r;
                if constexpr (has_cached_bounds<RangeF>::value) {
                    if (cached && cache.col_ready) r = range.cached(k, ci);
                    else r = range(k);
                } else {
                    r = range(k);
                }
                len = r.y - r.x;
                if (cached) {
                    if (!cache.col_ready) cache.col[ci] = k;
                    cache.bs[ci] = r.x;
                    cache.len[ci] = len;
                    if (VALUES && !cache.vals_ready) cache.av[ci] = av;
                }
            } else if (cached) {
                cache.bs[ci] = 0;
                cache.len[ci] = 0;
                if (VALUES) cache.av[ci] = 0.0;
            }
            if constexpr (ALIGNED) {
                // entry-aligned blocks: each entry rounds up to whole blocks
                const int nbc = __builtin_amdgcn_readlane(wave_incl_sum((len + kWave - 1) / kWave), kWave - 1);
                if (ln == 0) ctot[c] = nbc;
            } else {
                const int tot = __builtin_amdgcn_readlane(wave_incl_sum(len), kWave - 1);
                if (ln == 0) ctot[c] = (tot + kWave - 1) / kWave;
            }
        }
        if (threadIdx.x == 0) *claim = 0;
        __syncthreads();
        // 2. exclusive scan of the block counts. With fewer than 64 chunks (nearly every row) each wave scans
        //    them itself, in registers (lane i: the first block of chunk i; lane nch: the total), and no barrier
        //    is needed; otherwise wave 0 scans them into ctot (ctot[nch] = total blocks)
        const bool few = nch < kWave;
        int cpre = 0;
        if (few) {
            const int v = ln < nch ? ctot[ln] : 0;
            cpre = wave_incl_sum(v) - v;
        } else {
            if (wv == 0) {
                int carry = 0;
                for (int c0 = 0; c0 < nch; c0 += kWave) {
                    const int c = c0 + ln;
                    const int v = c < nch ? ctot[c] : 0;
                    const int inc = wave_incl_sum(v);
                    if (c < nch) ctot[c] = carry + inc - v;
                    carry += __builtin_amdgcn_readlane(inc, kWave - 1);
                }
                if (ln == 0) ctot[nch] = carry;
            }
            __syncthreads();
        }
        // first block of chunk i (i <= nch); i is uniform
        auto first_block = [&](int i) -> int {
            return few ? __builtin_amdgcn_readlane(cpre, i) : uniform(ctot[i]);
        };
        const int nb = first_block(nch);
        // a wave's chunk, held in registers, and its block range
        int c = -1, cb0 = 0, cb1 = 0;
        int boff = 0, len = 0, incl = 0, tot = 0;   // flattened blocks
        int bs = 0, bstart = 0, nblk = 0;            // entry-aligned blocks
        double av = 0.0;
        // processes blocks [b, e) of the group, moving forward through the chunks
        auto run = [&](int b, int e) {
            while (b < e) {
                if (b >= cb1) {
                    int cc = c < 0 ? 0 : c;
                    while (first_block(cc + 1) <= b) ++cc;
                    c = cc;
                    cb0 = first_block(c);
                    cb1 = first_block(c + 1);
                    const int a = g0 + c * kWave + ln;
                    bs = 0;
                    len = 0;
                    av = 0.0;
                    if (use_cache && c < kCacheChunks) {
                        const int ci = c * kWave + ln;
                        bs = cache.bs[ci];
                        len = cache.len[ci];
                        if (VALUES) av = cache.av[ci];
                    } else if (a < g1) {
                        const int2 r = range(a_col[a]);
                        bs = r.x;
                        len = r.y - r.x;
                        if (VALUES) av = to_d(a_val[a]);
                    }
                    if constexpr (ALIGNED) {
                        nblk = (len + kWave - 1) / kWave;
                        bstart = wave_incl_sum(nblk) - nblk;
                    } else {
                        incl = wave_incl_sum(len);
                        tot = __builtin_amdgcn_readlane(incl, kWave - 1);
                        boff = bs - (incl - len);
                    }
                }
                const int ee = cb1 < e ? cb1 : e;
                if constexpr (ALIGNED)
                    chunk_blocks_aligned<V, VALUES>(bs, av, len, bstart, nblk, b - cb0, ee - cb0, b_col, b_val, visit);
                else
                    chunk_blocks<V, VALUES, LONG, OFF32>(boff, av, len, incl, tot, b - cb0, ee - cb0, b_col, b_val, mark,
                                                  visit);
                b = ee;
            }
        };
        if constexpr (LONG) {
            // 3. claimed runs of blocks, guided: a claim takes about 1/(2 NW) of what was left at the wave's
            //    previous claim (a multiple of kUnitBlocks, at least kUnitBlocks), so claims are few while much
            //    remains and small near the end, where the last wave to finish sets the pass's time
            int seen = 0;   // claim position this wave saw last
            while (true) {
                int sz = (nb - seen) / (2 * NW);
                sz = (sz + kUnitBlocks - 1) / kUnitBlocks * kUnitBlocks;
                if (sz < kUnitBlocks) sz = kUnitBlocks;
                int b = 0;
                if (ln == 0) b = atomicAdd(claim, sz);
                b = uniform(b);
                if (b >= nb) break;
                seen = b + sz;
                run(b, nb - b < sz ? nb : b + sz);
            }
        } else {
            // 3. this wave's even share of the blocks
            const int b0 = static_cast<int>(static_cast<int64_t>(nb) * wv / NW);
            const int b1 = static_cast<int>(static_cast<int64_t>(nb) * (wv + 1) / NW);
            if (b0 < b1) {
                // last chunk whose first block is <= b0
                int lo = 0, hi = nch - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (first_block(mid) <= b0) lo = mid;
                    else hi = mid - 1;
                }
                c = lo;   // run() searches forward from here
                run(b0, b1);
            }
        }
        __syncthreads();
    }
}

}  // namespace wsp
