// Host orchestration and C ABI of the gfx950 SpGEMM (see include/wingspan.h).
//
// Symbolic phase: count the products of every row of A (a scan over A's
// entries of the lengths of the B rows they select), bin the rows by tier,
// run each tier's symbolic kernel to get the entry count of every row of C,
// and scan the counts into C.row_ptr.
// Numeric phase: bin the rows again from C.row_ptr, then run each tier's
// numeric kernel, which accumulates the row in its workspace and writes the
// row's columns (sorted) and values.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/wingspan.h"
#include "analysis.hpp"
#include "device_common.hpp"
#include "tiers.hpp"
#include "elementwise.hpp"
#include "spmspv.hpp"
#include "outer.hpp"

using namespace wsp;

namespace {

// ---------------------------------------------------------------------------
// Limits and defaults.
// ---------------------------------------------------------------------------
constexpr int kHashLog2MaxSym = 14;           // 16K int32 keys = 64 KB of LDS
constexpr int kHashLog2MaxNum = 13;           // 8K keys + 8K doubles = 96 KB of LDS
constexpr int64_t kBitmapMaxCols = 36864 * 32; // 144 KB LDS bitmap (plus per-wave marks)
constexpr int kMaxWindows = 128;              // dense numeric tier: windows per row
constexpr int64_t kStructCacheBytes = int64_t(4) << 30;   // default budget of the dense-row bitmaps kept from
                                                           // the symbolic to the numeric phase
// With the structure cache, rows from this many entries (products, in the symbolic phase) up take the
// bitmap / rank-indexed path even when they would fit an LDS hash table: the symbolic bitmap kernel is
// cheaper than a large LDS hash, and the rank-indexed numeric kernel, which then skips its structure
// pass, cheaper than a numeric hash table of 2^12 slots or more.
constexpr int64_t kCachedDenseMin = 2048;
// The single pass (no cache) sends rows from this many products up to the rank kernel when B's columns fit
// one of its regions: its structure pass is then one bitmap pass, cheaper than an LDS hash table sized by
// the row's products. Where B is wider a row is counted region by region first, and the LDS hash stays the
// cheaper tier wherever it fits.
constexpr int64_t kShardedDenseMin = 2048;
// With the structure cache and B's columns in one rank region, the symbolic phase already sends rows from
// this many products up to the bitmap kernel: below kCachedDenseMin they go back to the LDS hash in the
// numeric phase, but counting them in a bitmap costs less than in a hash table of 2^11 slots or more.
constexpr int64_t kSymbolicDenseMin = 1024;
constexpr int kDefaultWindow = 16384;         // 16K doubles = 128 KB of LDS
constexpr int64_t kPoolBytes = int64_t(1) << 30;   // spill pool: at most this, unless one table needs more
constexpr int64_t kMaxSlabCap = int64_t(1) << 27;
constexpr int kMaxSlabs = 256;                      // largest tables the pool holds at once (at most)
constexpr int64_t kMaxSpillGrid = 8192;             // spill workgroups per size class at most
constexpr size_t kAlign = 256;

thread_local std::string g_err;
thread_local wingspan_phase_stats g_stats[3];   // symbolic, numeric, single pass

wingspan_status fail(wingspan_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

#define HIP_TRY(call)                                                                     \
    do {                                                                                  \
        hipError_t e_ = (call);                                                           \
        if (e_ != hipSuccess)                                                             \
            return fail(WINGSPAN_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
    } while (0)

#define LAUNCH_CHECK(what)                                                                 \
    do {                                                                                   \
        hipError_t e_ = hipGetLastError();                                                 \
        if (e_ != hipSuccess)                                                              \
            return fail(WINGSPAN_ERR_HIP, "launch of %s failed: %s", what, hipGetErrorString(e_)); \
    } while (0)

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int64_t next_pow2(int64_t x) {
    int64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

struct Opts {
    bool validate = false;
    bool force_spill = false;
    bool timing = false;
    bool wide_offsets = false;
    bool dense_disabled = false;
    int hash_log2_max_sym = kHashLog2MaxSym;
    int hash_log2_max_num = kHashLog2MaxNum;
    int wcols = kDefaultWindow;
    bool wcols_explicit = false;   // window_cols given: use the column-window dense kernel
    int tiny_max = 64;
    int64_t dense_min_nnz = INT64_MAX;
    bool dense_min_explicit = false;   // dense_min_nnz given (otherwise chosen from the layout)
    int64_t cache_bytes = kStructCacheBytes;   // structure cache budget
};

wingspan_status parse_opts(const wingspan_options *o, Opts *out) {
    Opts r;
    if (o) {
        if (o->version != WINGSPAN_ABI_VERSION)
            return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "options->version is %u, expected %d", o->version,
                        WINGSPAN_ABI_VERSION);
        r.validate = o->validate != 0;
        r.force_spill = o->force_spill != 0;
        r.timing = o->timing != 0;
        r.wide_offsets = o->wide_offsets != 0;
        if (o->max_lds_slots != 0) {
            const int32_t s = o->max_lds_slots;
            if (s < 64 || s > (1 << 14) || (s & (s - 1)) != 0)
                return fail(WINGSPAN_ERR_INVALID_ARGUMENT,
                            "options->max_lds_slots must be a power of two in [64, 16384], got %d", s);
            const int l = ceil_log2(s);
            r.hash_log2_max_sym = std::min(r.hash_log2_max_sym, l);
            r.hash_log2_max_num = std::min(r.hash_log2_max_num, l);
        }
        if (o->window_cols != 0) {
            if (o->window_cols != 1024 && o->window_cols != 4096 && o->window_cols != 8192 &&
                o->window_cols != 16384)
                return fail(WINGSPAN_ERR_INVALID_ARGUMENT,
                            "options->window_cols must be 1024, 4096, 8192 or 16384, got %d", o->window_cols);
            r.wcols = o->window_cols;
            r.wcols_explicit = true;
        }
        if (o->tiny_max != 0) {
            if (o->tiny_max == -1) r.tiny_max = 0;
            else if (o->tiny_max < 8 || o->tiny_max > 64)
                return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "options->tiny_max must be -1 or in [8, 64], got %d",
                            o->tiny_max);
            else r.tiny_max = o->tiny_max;
        }
        if (o->dense_min_nnz == -1) r.dense_disabled = true;
        else if (o->dense_min_nnz < -1)
            return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "options->dense_min_nnz must be >= -1");
        else if (o->dense_min_nnz > 0) {
            r.dense_min_nnz = o->dense_min_nnz;
            r.dense_min_explicit = true;
        }
        if (o->cache_mib == -1) r.cache_bytes = 0;
        else if (o->cache_mib < -1)
            return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "options->cache_mib must be >= -1, got %d", o->cache_mib);
        else if (o->cache_mib > 0) r.cache_bytes = static_cast<int64_t>(o->cache_mib) << 20;
    }
    *out = r;
    return WINGSPAN_OK;
}

wingspan_status check_csr_desc(const wingspan_csr *M, const char *name) {
    if (!M) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (M->nrows < 0 || M->ncols < 0 || M->nnz < 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "%s has a negative dimension or nnz", name);
    if (M->nrows > INT32_MAX - 1 || M->ncols > INT32_MAX || M->nnz > INT32_MAX)
        return fail(WINGSPAN_ERR_INDEX_OVERFLOW, "%s exceeds the int32 index range", name);
    if (!M->row_ptr) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "%s->row_ptr is NULL", name);
    if (M->nnz > 0 && (!M->col_idx || !M->val))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "%s has nnz > 0 but a NULL col_idx or val", name);
    return WINGSPAN_OK;
}

wingspan_status check_pair(const wingspan_csr *A, const wingspan_csr *B) {
    wingspan_status s = check_csr_desc(A, "A");
    if (s != WINGSPAN_OK) return s;
    s = check_csr_desc(B, "B");
    if (s != WINGSPAN_OK) return s;
    if (A->ncols != B->nrows)
        return fail(WINGSPAN_ERR_DIMENSION_MISMATCH, "A.ncols (%lld) != B.nrows (%lld)",
                    (long long)A->ncols, (long long)B->nrows);
    return WINGSPAN_OK;
}

// Workspace layout, a pure function of the sizes and options.
struct Layout {
    size_t off_stamp, off_ctrl, off_pref, off_row_nnz, off_perm, off_rrows, off_partials, off_wtab, off_pool, total;
    size_t off_slot, off_cache;   // structure cache (cache_rows == 0: none)
    size_t off_ctrl_num, off_perm_num;   // the numeric binning kept from the symbolic phase (with the cache)
    int64_t row_words, cache_rows;
    int nwin;          // numeric dense windows per row (0: dense numeric tier unavailable)
    int wcols;         // columns per window of the window table
    bool rank_mode;    // dense numeric rows use the rank-indexed kernel
    int64_t slab_cap;    // slots of the largest spill table (a row beyond slab_cap / 2 entries is refused)
    int64_t pool_bytes;  // the spill pool
};

// budget > 0: the layout must fit `budget` bytes (the static scratch of the
// entry point that allocates nothing): no structure cache, and the spill pool
// takes what the other arrays leave, at least one slab. total > budget means
// the problem does not fit.
Layout plan(const wingspan_csr *A, const wingspan_csr *B, const Opts &o, size_t budget = 0) {
    Layout L{};
    const int64_t m = A->nrows, n = B->ncols, nnz_a = A->nnz;
    size_t off = 0;
    L.off_stamp = off;
    off += align_up(sizeof(Stamp));
    L.off_ctrl = off;
    off += align_up(sizeof(Control));
    L.off_ctrl_num = off;   // next to the stamp and the control block: the three are read back in one copy
    off += align_up(sizeof(Control));
    L.off_pref = off;
    off += align_up(sizeof(int64_t) * (nnz_a + 1));
    L.off_row_nnz = off;
    off += align_up(sizeof(int32_t) * std::max<int64_t>(m, 1));
    L.off_perm = off;
    off += align_up(sizeof(int32_t) * std::max<int64_t>(m, 1));
    L.off_rrows = off;
    off += align_up(sizeof(RankRow) * std::max<int64_t>(m, 1));
    L.off_partials = off;
    const int64_t tiles = (std::max<int64_t>(nnz_a, m + 1) + kScanTile - 1) / kScanTile + 2;
    off += align_up(sizeof(int64_t) * tiles);
    L.off_wtab = off;
    auto windows = [n](int64_t w) { return n > 0 ? (n + w - 1) / w : int64_t(1); };
    L.rank_mode = false;
    L.wcols = o.wcols;
    if (!o.wcols_explicit && windows(kRankWinCols) <= kMaxWindows) {
        L.rank_mode = true;
        L.wcols = kRankWinCols;
    }
    const int64_t nwin = windows(L.wcols);
    L.nwin = (!o.dense_disabled && nwin <= kMaxWindows) ? static_cast<int>(nwin) : 0;
    if (L.nwin > 0) off += align_up(sizeof(int32_t) * B->nrows * (L.nwin + 1) + sizeof(int32_t));
    L.off_pool = off;
    L.slab_cap = std::min(kMaxSlabCap, std::max<int64_t>(64, next_pow2(2 * std::max<int64_t>(n, 1))));
    const int64_t slab_bytes = L.slab_cap * 12;
    L.pool_bytes = std::max<int64_t>(slab_bytes, std::min<int64_t>(kPoolBytes, kMaxSlabs * slab_bytes));
    if (budget > 0) {
        const int64_t left = budget > off ? static_cast<int64_t>(budget - off) : 0;
        L.pool_bytes = std::max<int64_t>(slab_bytes, std::min<int64_t>(L.pool_bytes, left / 256 * 256));
    }
    off += align_up(static_cast<size_t>(L.pool_bytes));
    // structure cache: the symbolic phase's column bitmaps of dense rows, reused by the rank-indexed numeric
    // kernel; rows beyond the budget (options.cache_mib) run their own structure pass
    L.cache_rows = 0;
    L.row_words = 0;
    if (budget == 0 && L.rank_mode && L.nwin > 0 && !o.dense_disabled && n > 0 && n <= kBitmapMaxCols && m > 0) {
        L.row_words = (n + 31) / 32;
        L.row_words = (L.row_words + 63) / 64 * 64;
        L.cache_rows = std::min<int64_t>(m, o.cache_bytes / (L.row_words * 4));
    }
    L.off_perm_num = off;
    if (L.cache_rows > 0) off += align_up(sizeof(int32_t) * m);
    L.off_slot = off;
    if (L.cache_rows > 0) off += align_up(sizeof(int32_t) * m);
    L.off_cache = off;
    if (L.cache_rows > 0) off += align_up(static_cast<size_t>(L.cache_rows) * L.row_words * 4);
    L.total = off;
    return L;
}

// ---------------------------------------------------------------------------
// Per-call context.
// ---------------------------------------------------------------------------
struct Ctx {
    hipStream_t st;
    int dtype_f64 = -1;   // numeric value type: 1 double, 0 float, -1 unknown (symbolic)
    Opts o;
    Layout L;
    char *ws;
    Control *ctrl;
    int64_t *pref;
    int32_t *row_nnz;
    int32_t *perm;
    RankRow *rrows;
    int64_t *partials;
    int32_t *wtab;
    char *pool;
    Stamp *stamp;
    int32_t *slot_of_row;
    uint32_t *cache;
    Control *ctrl_num;        // the numeric binning the symbolic phase kept (with the cache)
    int32_t *perm_num;
    const int32_t *bins;      // numeric phase: the row ids grouped by bin it uses (perm or perm_num)
    bool wtab_ready = false;  // numeric phase: the window table is the one the symbolic phase built
    bool rrows_ready = false; // numeric phase: the dense rows' descriptions are the symbolic phase's
    bool side_ok = true;      // the numeric phase may run the light tiers on this thread's side stream
    Control host;
    Stamp host_stamp;
};

void carve(Ctx &c, void *ws) {
    c.ws = static_cast<char *>(ws);
    c.ctrl = reinterpret_cast<Control *>(c.ws + c.L.off_ctrl);
    c.pref = reinterpret_cast<int64_t *>(c.ws + c.L.off_pref);
    c.row_nnz = reinterpret_cast<int32_t *>(c.ws + c.L.off_row_nnz);
    c.perm = reinterpret_cast<int32_t *>(c.ws + c.L.off_perm);
    c.rrows = reinterpret_cast<RankRow *>(c.ws + c.L.off_rrows);
    c.partials = reinterpret_cast<int64_t *>(c.ws + c.L.off_partials);
    c.wtab = reinterpret_cast<int32_t *>(c.ws + c.L.off_wtab);
    c.pool = c.ws + c.L.off_pool;
    c.stamp = reinterpret_cast<Stamp *>(c.ws + c.L.off_stamp);
    c.slot_of_row = reinterpret_cast<int32_t *>(c.ws + c.L.off_slot);
    c.cache = reinterpret_cast<uint32_t *>(c.ws + c.L.off_cache);
    c.ctrl_num = reinterpret_cast<Control *>(c.ws + c.L.off_ctrl_num);
    c.perm_num = reinterpret_cast<int32_t *>(c.ws + c.L.off_perm_num);
    c.bins = c.perm;
}

// The stamp a symbolic phase on (A, B) with this layout leaves (magic and
// rp_sum are filled in on the device).
Stamp make_stamp(const Ctx &c, const wingspan_csr *A, const wingspan_csr *B, int64_t cached_rows = 0) {
    Stamp t{};
    t.cached_rows = cached_rows;
    t.a_rp = reinterpret_cast<uint64_t>(A->row_ptr);
    t.a_col = reinterpret_cast<uint64_t>(A->col_idx);
    t.b_rp = reinterpret_cast<uint64_t>(B->row_ptr);
    t.b_col = reinterpret_cast<uint64_t>(B->col_idx);
    t.a_nrows = A->nrows;
    t.a_ncols = A->ncols;
    t.a_nnz = A->nnz;
    t.b_nrows = B->nrows;
    t.b_ncols = B->ncols;
    t.b_nnz = B->nnz;
    t.off_slot = static_cast<int64_t>(c.L.off_slot);
    t.off_cache = static_cast<int64_t>(c.L.off_cache);
    t.row_words = c.L.row_words;
    t.cache_rows = c.L.cache_rows;
    return t;
}

// How the numeric phase bins rows (by C's exact row counts).
BinCfg numeric_bin_cfg(const Ctx &c, const wingspan_csr *B) {
    BinCfg cfg{};
    cfg.ncols = B->ncols;
    cfg.numeric = 1;
    cfg.tiny_max = c.o.tiny_max;
    cfg.force_spill = c.o.force_spill;
    cfg.hash_log2_max = c.o.hash_log2_max_num;
    cfg.dense_min_nnz = c.o.dense_min_nnz;
    cfg.dense_ok = c.L.nwin > 0;
    return cfg;
}

void stamp_bins(Stamp &t, const BinCfg &cfg, bool wtab) {
    t.num_bins = 1;
    t.wtab = wtab ? 1 : 0;
    t.nb_dense_min_nnz = cfg.dense_min_nnz;
    t.nb_tiny_max = cfg.tiny_max;
    t.nb_hash_log2_max = cfg.hash_log2_max;
    t.nb_force_spill = cfg.force_spill;
    t.nb_dense_ok = cfg.dense_ok;
}

// Whether the numeric phase may use the structure cache: the stamp is valid,
// was made for these inputs and this layout, and for the C.row_ptr given.
bool stamp_matches(const Ctx &c, const wingspan_csr *A, const wingspan_csr *B) {
    if (c.L.cache_rows <= 0) return false;
    const Stamp &h = c.host_stamp;
    const Stamp t = make_stamp(c, A, B);
    return h.magic == kStampMagic && h.a_rp == t.a_rp && h.a_col == t.a_col && h.b_rp == t.b_rp &&
           h.b_col == t.b_col && h.a_nrows == t.a_nrows && h.a_ncols == t.a_ncols && h.a_nnz == t.a_nnz &&
           h.b_nrows == t.b_nrows && h.b_ncols == t.b_ncols && h.b_nnz == t.b_nnz && h.off_slot == t.off_slot &&
           h.off_cache == t.off_cache && h.row_words == t.row_words && h.cache_rows == t.cache_rows &&
           h.rp_sum == c.host.rp_sum;
}

// HIP events for optional per-tier timing, created once per thread.
struct Timer {
    bool on = false;
    hipEvent_t ev[2 * (WINGSPAN_NUM_TIERS + 1)] = {};
    bool made = false;
};
thread_local Timer g_timer;

wingspan_status timer_start(Ctx &c, int slot) {
    if (!g_timer.on) return WINGSPAN_OK;
    HIP_TRY(hipEventRecord(g_timer.ev[2 * slot], c.st));
    return WINGSPAN_OK;
}
wingspan_status timer_stop(Ctx &c, int slot) {
    if (!g_timer.on) return WINGSPAN_OK;
    HIP_TRY(hipEventRecord(g_timer.ev[2 * slot + 1], c.st));
    return WINGSPAN_OK;
}

wingspan_status timer_begin(bool on) {
    g_timer.on = on;
    if (on && !g_timer.made) {
        for (auto &e : g_timer.ev) HIP_TRY(hipEventCreate(&e));
        g_timer.made = true;
    }
    return WINGSPAN_OK;
}

constexpr int kSlotAnalysis = WINGSPAN_NUM_TIERS;

// A second stream per thread and device (default priority) with a fork and a
// join event, so the numeric phase's light tiers can run beside the dense
// kernel: they start where the dense kernel's workgroups leave CUs free.
struct SideStream {
    int dev = -1;
    hipStream_t st = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};
thread_local std::vector<SideStream> g_side;

wingspan_status side_stream(SideStream **out) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    for (SideStream &s : g_side)
        if (s.dev == dev) {
            *out = &s;
            return WINGSPAN_OK;
        }
    SideStream s;
    s.dev = dev;
    HIP_TRY(hipStreamCreateWithFlags(&s.st, hipStreamNonBlocking));
    HIP_TRY(hipEventCreateWithFlags(&s.fork, hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&s.join, hipEventDisableTiming));
    g_side.push_back(s);
    *out = &g_side.back();
    return WINGSPAN_OK;
}

template <typename In>
wingspan_status run_scan(Ctx &c, In in, int64_t n, int64_t *out) {
    const int64_t nb = std::max<int64_t>(1, (n + kScanTile - 1) / kScanTile);
    scan_tile_sums<In><<<dim3(static_cast<unsigned>(nb)), kScanBlock, 0, c.st>>>(in, n, c.partials);
    scan_partials<<<1, 1024, 0, c.st>>>(c.partials, nb);
    scan_tiles<In><<<dim3(static_cast<unsigned>(nb)), kScanBlock, 0, c.st>>>(in, n, c.partials, nb, out);
    LAUNCH_CHECK("scan");
    return WINGSPAN_OK;
}

unsigned blocks_for(int64_t n, int per) { return static_cast<unsigned>((n + per - 1) / per); }

// Product counts, optional validation, and binning. Ends with the control
// block on the host.
// What the analysis prepares: the symbolic phase (bins by products, LDS
// tables of keys), the numeric phase (bins by C's exact row counts), or the
// single pass with sharded output (bins by products, LDS tables of keys and
// doubles; row_nnz_out receives 0 for the rows without products).
enum AnalysisMode { kModeSymbolic = 0, kModeNumeric = 1, kModeSharded = 2 };

wingspan_status analyze(Ctx &c, const wingspan_csr *A, const wingspan_csr *B, AnalysisMode mode,
                        const int64_t *c_rp, bool have_pref, int32_t *row_nnz_out = nullptr) {
    wingspan_status s;
    const bool numeric = mode == kModeNumeric;
    if ((s = timer_start(c, kSlotAnalysis)) != WINGSPAN_OK) return s;
    const int64_t m = A->nrows;
    const int64_t words = sizeof(Control) / sizeof(int32_t);
    zero_words<<<blocks_for(words, 256), 256, 0, c.st>>>(reinterpret_cast<int32_t *>(c.ctrl), words);
    LAUNCH_CHECK("zero_words");
    c.bins = c.perm;
    c.wtab_ready = false;
    c.rrows_ready = false;
    if (numeric && c.L.cache_rows > 0 && !c.o.validate) {
        // The symbolic phase on the same workspace may have binned the rows by this C.row_ptr already: check
        // its stamp (with C.row_ptr's checksum) and take its bins if they were made with these settings
        rowptr_checksum<<<64, 256, 0, c.st>>>(c_rp, m, &c.ctrl->rp_sum);
        LAUNCH_CHECK("stamp");
        // the stamp, the control block and the kept binning, adjacent in the workspace, in one copy
        static_assert(sizeof(Stamp) <= kAlign * 2, "stamp region");
        const size_t span = c.L.off_ctrl_num + sizeof(Control) - c.L.off_stamp;
        thread_local std::vector<char> back;
        back.resize(span);
        HIP_TRY(hipMemcpyAsync(back.data(), c.ws + c.L.off_stamp, span, hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
        Control kept;
        std::memcpy(&c.host_stamp, back.data(), sizeof(Stamp));
        std::memcpy(&c.host, back.data() + (c.L.off_ctrl - c.L.off_stamp), sizeof(Control));
        std::memcpy(&kept, back.data() + (c.L.off_ctrl_num - c.L.off_stamp), sizeof(Control));
        const BinCfg cfg = numeric_bin_cfg(c, B);
        const Stamp &h = c.host_stamp;
        if (stamp_matches(c, A, B) && h.num_bins == 1 && h.nb_dense_min_nnz == cfg.dense_min_nnz &&
            h.nb_tiny_max == cfg.tiny_max && h.nb_hash_log2_max == cfg.hash_log2_max &&
            h.nb_force_spill == cfg.force_spill && h.nb_dense_ok == cfg.dense_ok) {
            const uint64_t rp_sum = c.host.rp_sum;
            c.host = kept;
            c.host.rp_sum = rp_sum;
            c.bins = c.perm_num;
            c.wtab_ready = h.wtab == 1;
            c.rrows_ready = h.wtab == 1;   // built with the window table
            if ((s = timer_stop(c, kSlotAnalysis)) != WINGSPAN_OK) return s;
            const int64_t slab_limit = c.L.slab_cap / 2;
            if (c.host.spill_max_bound > slab_limit)
                return fail(WINGSPAN_ERR_UNSUPPORTED,
                            "a row needs %lld hash slots but the spill pool's slabs hold %lld entries",
                            (long long)c.host.spill_max_bound, (long long)slab_limit);
            return WINGSPAN_OK;
        }
        // not kept for this call: bin here (the checksum is added again below)
        zero_words<<<blocks_for(words, 256), 256, 0, c.st>>>(reinterpret_cast<int32_t *>(c.ctrl), words);
        LAUNCH_CHECK("zero_words");
    }
    if (mode == kModeSymbolic || mode == kModeSharded) {
        // the structure cache (and what the symbolic phase keeps for the numeric one) is being rewritten:
        // invalid until a symbolic phase completes
        write_stamp<<<1, 1, 0, c.st>>>(c.stamp, Stamp{});
    } else if (numeric && c.L.cache_rows > 0) {
        rowptr_checksum<<<64, 256, 0, c.st>>>(c_rp, m, &c.ctrl->rp_sum);
    }
    LAUNCH_CHECK("stamp");
    if (c.o.validate) {
        if (A->nrows > 0)
            validate_csr<<<blocks_for(A->nrows * kWave, 256), 256, 0, c.st>>>(A->row_ptr, A->col_idx, A->nrows,
                                                                             A->ncols, A->nnz, c.ctrl);
        if (B->nrows > 0)
            validate_csr<<<blocks_for(B->nrows * kWave, 256), 256, 0, c.st>>>(B->row_ptr, B->col_idx, B->nrows,
                                                                             B->ncols, B->nnz, c.ctrl);
        LAUNCH_CHECK("validate_csr");
        // the product counts below index B.row_ptr through A.col_idx: stop
        // here if the inputs are not canonical
        HIP_TRY(hipMemcpyAsync(&c.host, c.ctrl, sizeof(Control), hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
        if (c.host.error_flags & kErrInvalidMatrix)
            return fail(WINGSPAN_ERR_INVALID_MATRIX, "A or B is not canonical CSR");
    }
    if (!have_pref) {
        s = run_scan(c, BRowLenIn{A->col_idx, B->row_ptr}, A->nnz, c.pref);
        if (s != WINGSPAN_OK) return s;
    }
    if (numeric && c.dtype_f64 >= 0 && !c.L.rank_mode) {
        // only the column-window dense kernel's sentinel slots depend on it
        const unsigned zb = 1024;
        if (c.dtype_f64) {
            find_zero_values<double><<<zb, 256, 0, c.st>>>(static_cast<const double *>(A->val), A->nnz, c.ctrl);
            if (B->val != A->val)
                find_zero_values<double><<<zb, 256, 0, c.st>>>(static_cast<const double *>(B->val), B->nnz, c.ctrl);
        } else {
            find_zero_values<float><<<zb, 256, 0, c.st>>>(static_cast<const float *>(A->val), A->nnz, c.ctrl);
            if (B->val != A->val)
                find_zero_values<float><<<zb, 256, 0, c.st>>>(static_cast<const float *>(B->val), B->nnz, c.ctrl);
        }
        LAUNCH_CHECK("find_zero_values");
    }
    BinCfg cfg{};
    cfg.ncols = B->ncols;
    cfg.numeric = numeric;
    cfg.tiny_max = c.o.tiny_max;
    cfg.force_spill = c.o.force_spill;
    cfg.hash_log2_max = mode == kModeSymbolic ? c.o.hash_log2_max_sym : c.o.hash_log2_max_num;
    cfg.dense_min_nnz = c.o.dense_min_nnz;
    if (mode == kModeNumeric) {
        cfg = numeric_bin_cfg(c, B);
    } else if (mode == kModeSymbolic) {
        cfg.dense_ok = !c.o.dense_disabled && B->ncols <= kBitmapMaxCols;
        if (!c.o.dense_min_explicit && c.L.cache_rows > 0 && B->ncols <= RankShape<float>::REGION_COLS)
            cfg.dense_min_nnz = kSymbolicDenseMin;
    } else {
        // the rank kernel writes a pool row once its count is known (a row of several regions counts them
        // first)
        cfg.dense_ok = c.L.rank_mode && c.L.nwin > 0;
        cfg.dense_min_nnz = c.o.dense_min_explicit
                                ? c.o.dense_min_nnz
                                : (B->ncols <= RankShape<float>::REGION_COLS ? kShardedDenseMin : INT64_MAX);
    }
    if (m > 0) {
        bin_count<<<blocks_for(m, 256), 256, 0, c.st>>>(A->row_ptr, c.pref, c_rp, m, cfg, c.ctrl,
                                                         row_nnz_out ? row_nnz_out : c.row_nnz);
        bin_offsets<<<1, 1, 0, c.st>>>(c.ctrl, c.pref, A->nnz);
        bin_scatter<<<blocks_for(m, 256), 256, 0, c.st>>>(A->row_ptr, c.pref, c_rp, m, cfg, c.ctrl, c.perm);
    } else {
        bin_offsets<<<1, 1, 0, c.st>>>(c.ctrl, c.pref, A->nnz);
    }
    LAUNCH_CHECK("binning");
    if ((s = timer_stop(c, kSlotAnalysis)) != WINGSPAN_OK) return s;
    HIP_TRY(hipMemcpyAsync(&c.host, c.ctrl, sizeof(Control), hipMemcpyDeviceToHost, c.st));
    if (numeric && c.L.cache_rows > 0)
        HIP_TRY(hipMemcpyAsync(&c.host_stamp, c.stamp, sizeof(Stamp), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    const int64_t slab_limit = c.L.slab_cap / 2;
    if (c.host.spill_max_bound > slab_limit)
        return fail(WINGSPAN_ERR_UNSUPPORTED,
                    "a row needs %lld hash slots but the spill pool's slabs hold %lld entries",
                    (long long)c.host.spill_max_bound, (long long)slab_limit);
    return WINGSPAN_OK;
}

int tier_of_bin(int b) {
    if (b >= kBinTiny0 && b < kBinTiny0 + kNumTiny) return WINGSPAN_TIER_TINY;
    if (b >= kBinHash0 && b < kBinHash0 + kNumHash) return WINGSPAN_TIER_HASH;
    if (b >= kBinDense0 && b < kBinDense0 + kNumClasses) return WINGSPAN_TIER_DENSE;
    if (b >= kBinSpill0 && b < kBinSpill0 + kNumClasses) return WINGSPAN_TIER_SPILL;
    return -1;
}

void fill_stats(const Ctx &c, int phase) {
    wingspan_phase_stats &st = g_stats[phase];
    st = wingspan_phase_stats{};
    for (int b = 0; b < kNumBins; ++b) {
        const int t = tier_of_bin(b);
        if (t < 0) continue;
        st.rows[t] += c.host.bin_count[b];
        st.a_nnz[t] += c.host.stat_annz[b];
        st.products[t] += c.host.stat_products[b];
        st.c_nnz[t] += c.host.stat_cnnz[b];
    }
    st.total_products = c.host.total_products;
}

// Whether every byte offset of B's columns and values fits in 32 bits, so the
// rank kernel may form its B offsets in 32 bits.
template <typename V>
bool offsets_fit_32(const wingspan_csr *B) {
    return B->nnz <= (int64_t(1) << 32) / static_cast<int64_t>(sizeof(V));
}

// Workgroups of the persistent rank kernel: one per compute unit of the
// current device (its LDS use allows no second), or fewer when there are fewer
// rows.
unsigned rank_grid(int32_t rows) {
    static int cus[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
    if (cus[dev] <= 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cus[dev] = n;
    }
    return static_cast<unsigned>(std::min<int32_t>(rows, cus[dev]));
}

// Contiguous range of perm covering bins [b0, b0+nb).
void bin_range(const Ctx &c, int b0, int nb, int32_t *start, int32_t *count) {
    *start = c.host.bin_offset[b0];
    int32_t cnt = 0;
    for (int b = b0; b < b0 + nb; ++b) cnt += c.host.bin_count[b];
    *count = cnt;
}

// ---------------------------------------------------------------------------
// Kernel dispatch over compile-time shapes.
// ---------------------------------------------------------------------------
template <typename V, bool NUM>
void launch_tiny(int s_idx, unsigned grid, hipStream_t st, const Mats<V> &M, const int32_t *rows,
                 int32_t cnt, int32_t *row_nnz, RowSink out, int32_t *c_col, V *c_val, Control *ctrl) {
    switch (s_idx) {
        case 0: tiny_kernel<8, V, NUM><<<grid, 256, 0, st>>>(M, rows, cnt, row_nnz, out, c_col, c_val, ctrl); break;
        case 1: tiny_kernel<16, V, NUM><<<grid, 256, 0, st>>>(M, rows, cnt, row_nnz, out, c_col, c_val, ctrl); break;
        case 2: tiny_kernel<32, V, NUM><<<grid, 256, 0, st>>>(M, rows, cnt, row_nnz, out, c_col, c_val, ctrl); break;
        default: tiny_kernel<64, V, NUM><<<grid, 256, 0, st>>>(M, rows, cnt, row_nnz, out, c_col, c_val, ctrl); break;
    }
}

template <int LOG2T, typename V, bool NUM>
void launch_hash_t(unsigned grid, hipStream_t st, const Mats<V> &M, const int32_t *rows, int64_t ncols,
                   int32_t *row_nnz, RowSink out, int32_t *c_col, V *c_val, Control *ctrl) {
    hash_kernel<LOG2T, V, NUM><<<grid, HashShape<LOG2T>::BLOCK, 0, st>>>(M, rows, ncols, row_nnz, out, c_col,
                                                                        c_val, ctrl);
}

template <typename V, bool NUM>
void launch_hash(int log2t, unsigned grid, hipStream_t st, const Mats<V> &M, const int32_t *rows, int64_t ncols,
                 int32_t *row_nnz, RowSink out, int32_t *c_col, V *c_val, Control *ctrl) {
#define WS_HASH_CASE(L) \
    case L: launch_hash_t<L, V, NUM>(grid, st, M, rows, ncols, row_nnz, out, c_col, c_val, ctrl); break;
    switch (log2t) {
        WS_HASH_CASE(6)
        WS_HASH_CASE(7)
        WS_HASH_CASE(8)
        WS_HASH_CASE(9)
        WS_HASH_CASE(10)
        WS_HASH_CASE(11)
        WS_HASH_CASE(12)
        WS_HASH_CASE(13)
        default:
            if constexpr (!NUM) launch_hash_t<14, V, NUM>(grid, st, M, rows, ncols, row_nnz, out, c_col, c_val, ctrl);
            break;
    }
#undef WS_HASH_CASE
}

void launch_bitmap(int64_t ncols, unsigned grid, hipStream_t st, const Mats<float> &M, const int32_t *rows,
                   int32_t *row_nnz, int32_t *slot_of_row, uint32_t *cache, int64_t row_words, int64_t cache_rows) {
    const int nwords = static_cast<int>((ncols + 31) / 32);
#define WS_BITMAP(NW, BL) \
    bitmap_sym_kernel<NW, BL><<<grid, BL, 0, st>>>(M, rows, nwords, row_nnz, slot_of_row, cache, row_words, cache_rows)
    if (nwords <= 2048) WS_BITMAP(2048, 512);
    else if (nwords <= 8192) WS_BITMAP(8192, 512);
    else if (nwords <= 16384) WS_BITMAP(16384, 1024);
    else if (nwords <= 32768) WS_BITMAP(32768, 1024);
    else WS_BITMAP(36864, 1024);
#undef WS_BITMAP
}

template <int WV, typename V>
void launch_dense_w(bool sentinel, unsigned grid, hipStream_t st, const Mats<V> &M, const int32_t *rows,
                    const int32_t *wtab, int nwin, int64_t ncols, const int64_t *c_rp, int32_t *c_col, V *c_val,
                    Control *ctrl) {
    constexpr int BLOCK = DenseShape<WV>::BLOCK;
    if (sentinel)
        dense_num_kernel<WV, V, true><<<grid, BLOCK, 0, st>>>(M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
    else
        dense_num_kernel<WV, V, false><<<grid, BLOCK, 0, st>>>(M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
}

template <typename V>
void launch_dense(int wcols, bool sentinel, unsigned grid, hipStream_t st, const Mats<V> &M, const int32_t *rows,
                  const int32_t *wtab, int nwin, int64_t ncols, const int64_t *c_rp, int32_t *c_col, V *c_val,
                  Control *ctrl) {
    if (wcols == 1024)
        launch_dense_w<1024, V>(sentinel, grid, st, M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
    else if (wcols == 4096)
        launch_dense_w<4096, V>(sentinel, grid, st, M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
    else if (wcols == 8192)
        launch_dense_w<8192, V>(sentinel, grid, st, M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
    else
        launch_dense_w<16384, V>(sentinel, grid, st, M, rows, wtab, nwin, ncols, c_rp, c_col, c_val, ctrl);
}

// The spill tier, one launch per size class (heaviest first). Class k holds
// rows with fewer than 2^(26-k) products (k >= 1; class 0 is unbounded), whose
// tables hold nextpow2(2 * min(products, ncols)) slots at most: the class's
// slabs are that size (or the largest table, slab_cap), and as many
// workgroups run as the pool holds slabs.
template <typename V, bool NUM>
wingspan_status launch_spill(Ctx &c, const Mats<V> &M, const int32_t *perm, int64_t ncols, int32_t *row_nnz,
                             const RowSink &out, int32_t *c_col, V *c_val, int32_t *launches) {
    for (int k = 0; k < kNumClasses; ++k) {
        const int b = kBinSpill0 + k;
        const int32_t cnt = c.host.bin_count[b];
        if (!cnt) continue;
        int64_t slab = c.L.slab_cap;
        if (k >= 1 && 26 - k < 62) slab = std::min<int64_t>(slab, std::max<int64_t>(64, int64_t(1) << (27 - k)));
        const int64_t fits = c.L.pool_bytes / (slab * 12);
        const unsigned grid = static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>({int64_t(cnt), fits,
                                                                                             kMaxSpillGrid})));
        spill_kernel<V, NUM><<<grid, kSpillBlock, 0, c.st>>>(M, perm + c.host.bin_offset[b], cnt, c.pref, ncols,
                                                             c.pool, slab, row_nnz, out, c_col, c_val, c.ctrl,
                                                             &c.ctrl->spill_next[k]);
        ++*launches;
        LAUNCH_CHECK("spill");
    }
    return WINGSPAN_OK;
}

// ---------------------------------------------------------------------------
// Phases.
// ---------------------------------------------------------------------------
wingspan_status symbolic_impl(Ctx &c, const wingspan_csr *A, const wingspan_csr *B, int64_t *c_rp,
                              int64_t *c_nnz) {
    wingspan_status s = analyze(c, A, B, kModeSymbolic, nullptr, false);
    if (s != WINGSPAN_OK) return s;
    fill_stats(c, 0);
    wingspan_phase_stats &stats = g_stats[0];
    const Mats<float> M{A->row_ptr, A->col_idx, static_cast<const float *>(A->val),
                        B->row_ptr, B->col_idx, static_cast<const float *>(B->val)};
    const int32_t *perm = c.perm;
    int32_t start, cnt;
    bin_range(c, kBinDense0, kNumClasses, &start, &cnt);
    const bool caching = c.L.cache_rows > 0;
    const int64_t cnt_dense = cnt;
    // B's window table for the numeric phase's dense rows (it depends on B only)
    const bool wtab = caching && cnt_dense > 0 && c.L.nwin > 0;
    int32_t light = 0;
    for (int b = kBinTiny0; b < kBinTiny0 + kNumTiny; ++b) light += c.host.bin_count[b];
    for (int b = kBinHash0; b < kBinHash0 + kNumHash; ++b) light += c.host.bin_count[b];
    // untimed, the tiny and hash tiers (and the window table) run on a side stream beside the dense kernel,
    // joined before the spill tier; timed, every tier runs in turn on the caller's stream
    SideStream *side = nullptr;
    if (!g_timer.on && c.side_ok && cnt && (light || wtab)) {
        if ((s = side_stream(&side)) != WINGSPAN_OK) return s;
        HIP_TRY(hipEventRecord(side->fork, c.st));
    }
    const hipStream_t light_st = side ? side->st : c.st;
    auto light_tiers = [&]() -> wingspan_status {
        if (side) HIP_TRY(hipStreamWaitEvent(side->st, side->fork, 0));
        if ((s = timer_start(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;
        for (int i = 0; i < kNumTiny; ++i) {
            const int b = kBinTiny0 + i;
            const int32_t nb = c.host.bin_count[b];
            if (!nb) continue;
            const int S = 8 << i;
            launch_tiny<float, false>(i, blocks_for(int64_t(nb) * S, 256), light_st, M, perm + c.host.bin_offset[b],
                                      nb, c.row_nnz, RowSink{}, nullptr, nullptr, c.ctrl);
            stats.launches[WINGSPAN_TIER_TINY]++;
        }
        LAUNCH_CHECK("tiny symbolic");
        if ((s = timer_stop(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;

        if ((s = timer_start(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;
        for (int i = 0; i < kNumHash; ++i) {
            const int b = kBinHash0 + i;
            const int32_t nb = c.host.bin_count[b];
            if (!nb) continue;
            launch_hash<float, false>(kHashLog2Min + i, static_cast<unsigned>(nb), light_st, M,
                                      perm + c.host.bin_offset[b], B->ncols, c.row_nnz, RowSink{}, nullptr, nullptr,
                                      c.ctrl);
            stats.launches[WINGSPAN_TIER_HASH]++;
        }
        LAUNCH_CHECK("hash symbolic");
        if ((s = timer_stop(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;
        if (wtab) {
            const int64_t entries = B->nrows * static_cast<int64_t>(c.L.nwin + 1);
            build_window_table<<<blocks_for(entries, 256), 256, 0, light_st>>>(B->row_ptr, B->col_idx, B->nrows,
                                                                               c.L.nwin, c.L.wcols, c.wtab);
            LAUNCH_CHECK("build_window_table");
        }
        if (side) HIP_TRY(hipEventRecord(side->join, side->st));
        return WINGSPAN_OK;
    };
    if (!side && (s = light_tiers()) != WINGSPAN_OK) return s;

    if ((s = timer_start(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;
    if (caching) {
        fill_i32<<<blocks_for(A->nrows, 256), 256, 0, c.st>>>(c.slot_of_row, A->nrows, -1);
        LAUNCH_CHECK("fill slots");
    }
    if (cnt) {
        launch_bitmap(B->ncols, static_cast<unsigned>(cnt), c.st, M, perm + start, c.row_nnz,
                      caching ? c.slot_of_row : nullptr, caching ? c.cache : nullptr, c.L.row_words,
                      c.L.cache_rows);
        stats.launches[WINGSPAN_TIER_DENSE]++;
        LAUNCH_CHECK("bitmap symbolic");
    }
    if ((s = timer_stop(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;
    if (side) {
        if ((s = light_tiers()) != WINGSPAN_OK) return s;
        HIP_TRY(hipStreamWaitEvent(c.st, side->join, 0));
    }

    if ((s = timer_start(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;
    s = launch_spill<float, false>(c, M, perm, B->ncols, c.row_nnz, RowSink{}, nullptr, nullptr,
                                   &stats.launches[WINGSPAN_TIER_SPILL]);
    if (s != WINGSPAN_OK) return s;
    if ((s = timer_stop(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;

    s = run_scan(c, CountIn{c.row_nnz}, A->nrows, c_rp);
    if (s != WINGSPAN_OK) return s;
    if (caching) {
        // C.row_ptr is known: bin the rows as the numeric phase does, and build B's window table for the dense
        // rows (the numeric phase's dense rows are symbolic dense rows too: a row's entries never exceed its
        // products), so a numeric phase on this workspace starts from them
        const BinCfg ncfg = numeric_bin_cfg(c, B);
        const int64_t words = sizeof(Control) / sizeof(int32_t);
        zero_words<<<blocks_for(words, 256), 256, 0, c.st>>>(reinterpret_cast<int32_t *>(c.ctrl_num), words);
        bin_count<<<blocks_for(A->nrows, 256), 256, 0, c.st>>>(A->row_ptr, c.pref, c_rp, A->nrows, ncfg, c.ctrl_num,
                                                                 c.row_nnz);
        bin_offsets<<<1, 1, 0, c.st>>>(c.ctrl_num, c.pref, A->nnz);
        bin_scatter<<<blocks_for(A->nrows, 256), 256, 0, c.st>>>(A->row_ptr, c.pref, c_rp, A->nrows, ncfg,
                                                                   c.ctrl_num, c.perm_num);
        LAUNCH_CHECK("numeric binning");
        if (wtab) {
            // (the window table was built beside the tiers) and the descriptions of the numeric phase's dense
            // rows (their cache slots are this phase's)
            rank_rows_of_bins<<<blocks_for(A->nrows, 256), 256, 0, c.st>>>(c.perm_num, c.ctrl_num, A->row_ptr, c_rp,
                                                                           c.slot_of_row, c.rrows);
            LAUNCH_CHECK("rank rows of bins");
        }
        // the cache is complete: stamp it with the inputs, the layout, the bins' settings and C.row_ptr's
        // checksum
        Stamp t = make_stamp(c, A, B, std::min<int64_t>(cnt_dense, c.L.cache_rows));
        stamp_bins(t, ncfg, wtab);
        write_stamp<<<1, 1, 0, c.st>>>(c.stamp, t);
        rowptr_checksum<<<64, 256, 0, c.st>>>(c_rp, A->nrows, &c.stamp->rp_sum);
        seal_stamp<<<1, 1, 0, c.st>>>(c.stamp);
        LAUNCH_CHECK("stamp");
    }
    int64_t total = 0;
    HIP_TRY(hipMemcpyAsync(&total, c_rp + A->nrows, sizeof(int64_t), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    *c_nnz = total;
    stats.c_nnz_total = total;
    return WINGSPAN_OK;
}

template <typename V>
wingspan_status numeric_impl(Ctx &c, const wingspan_csr *A, const wingspan_csr *B, const int64_t *c_rp,
                             int32_t *c_col, V *c_val, bool have_pref) {
    wingspan_status s = analyze(c, A, B, kModeNumeric, c_rp, have_pref);
    if (s != WINGSPAN_OK) return s;
    fill_stats(c, 1);
    wingspan_phase_stats &stats = g_stats[1];
    int64_t c_entries = 0;
    for (int b = 0; b < kNumBins; ++b) c_entries += c.host.stat_cnnz[b];
    stats.c_nnz_total = c_entries;
    if (c_entries > 0 && (!c_col || !c_val))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "C has %lld entries but c_col_idx_dev or c_val_dev is NULL",
                    (long long)c_entries);
    const Mats<V> M{A->row_ptr, A->col_idx, static_cast<const V *>(A->val),
                    B->row_ptr, B->col_idx, static_cast<const V *>(B->val)};
    const int32_t *perm = c.bins;
    RowSink sink;
    sink.c_rp = c_rp;

    int32_t start, cnt;
    bin_range(c, kBinDense0, kNumClasses, &start, &cnt);
    int32_t light = 0;
    for (int b = kBinTiny0; b < kBinTiny0 + kNumTiny; ++b) light += c.host.bin_count[b];
    for (int b = kBinHash0; b < kBinHash0 + kNumHash; ++b) light += c.host.bin_count[b];
    // untimed, the tiny and hash tiers run on a side stream beside the dense kernel (forked after the analysis,
    // joined before the spill tier); timed, every tier runs in turn on the caller's stream
    SideStream *side = nullptr;
    if (!g_timer.on && c.side_ok && cnt && light) {
        if ((s = side_stream(&side)) != WINGSPAN_OK) return s;
        HIP_TRY(hipEventRecord(side->fork, c.st));
    }
    const hipStream_t light_st = side ? side->st : c.st;
    auto light_tiers = [&]() -> wingspan_status {
        if (side) HIP_TRY(hipStreamWaitEvent(side->st, side->fork, 0));
        if ((s = timer_start(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;
        for (int i = 0; i < kNumTiny; ++i) {
            const int b = kBinTiny0 + i;
            const int32_t nb = c.host.bin_count[b];
            if (!nb) continue;
            const int S = 8 << i;
            launch_tiny<V, true>(i, blocks_for(int64_t(nb) * S, 256), light_st, M, perm + c.host.bin_offset[b], nb,
                                 nullptr, sink, c_col, c_val, c.ctrl);
            stats.launches[WINGSPAN_TIER_TINY]++;
        }
        LAUNCH_CHECK("tiny numeric");
        if ((s = timer_stop(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;

        if ((s = timer_start(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;
        for (int i = 0; i < kNumHash; ++i) {
            const int b = kBinHash0 + i;
            const int32_t nb = c.host.bin_count[b];
            if (!nb) continue;
            launch_hash<V, true>(kHashLog2Min + i, static_cast<unsigned>(nb), light_st, M, perm + c.host.bin_offset[b],
                                 B->ncols, nullptr, sink, c_col, c_val, c.ctrl);
            stats.launches[WINGSPAN_TIER_HASH]++;
        }
        LAUNCH_CHECK("hash numeric");
        if ((s = timer_stop(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;
        if (side) {
            HIP_TRY(hipEventRecord(side->join, side->st));
        }
        return WINGSPAN_OK;
    };
    if (!side && (s = light_tiers()) != WINGSPAN_OK) return s;

    if (cnt && !c.wtab_ready) {
        const int64_t entries = B->nrows * static_cast<int64_t>(c.L.nwin + 1);
        build_window_table<<<blocks_for(entries, 256), 256, 0, c.st>>>(B->row_ptr, B->col_idx, B->nrows, c.L.nwin,
                                                                       c.L.wcols, c.wtab);
        LAUNCH_CHECK("build_window_table");
    }
    // the dense tier's time covers its one kernel launch only
    if ((s = timer_start(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;
    if (cnt && c.L.rank_mode) {
        const bool cached = stamp_matches(c, A, B);
        stats.structure_cache_rows = cached ? c.host_stamp.cached_rows : 0;
        if (!c.rrows_ready || !cached)
            rank_rows<<<blocks_for(cnt, 256), 256, 0, c.st>>>(perm + start, cnt, A->row_ptr, c_rp,
                                                                cached ? c.slot_of_row : nullptr, c.rrows);
        LAUNCH_CHECK("rank rows");
        const uint32_t *cache = cached ? c.cache : nullptr;
        if (!c.o.wide_offsets && offsets_fit_32<V>(B))
            dense_rank_kernel<V, false, true><<<rank_grid(cnt), RankShape<V>::BLOCK, 0, c.st>>>(
                M, c.rrows, cnt, c.wtab, c.L.nwin, B->ncols, sink, c_col, c_val, c.ctrl, cache, c.L.row_words);
        else
            dense_rank_kernel<V, false, false><<<rank_grid(cnt), RankShape<V>::BLOCK, 0, c.st>>>(
                M, c.rrows, cnt, c.wtab, c.L.nwin, B->ncols, sink, c_col, c_val, c.ctrl, cache, c.L.row_words);
        stats.launches[WINGSPAN_TIER_DENSE]++;
        LAUNCH_CHECK("dense rank numeric");
    } else if (cnt) {
        launch_dense<V>(c.L.wcols, c.host.has_zero_values == 0, static_cast<unsigned>(cnt), c.st, M, perm + start,
                        c.wtab, c.L.nwin, B->ncols, c_rp, c_col, c_val, c.ctrl);
        stats.launches[WINGSPAN_TIER_DENSE]++;
        LAUNCH_CHECK("dense numeric");
    }
    if ((s = timer_stop(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;
    if (side) {
        if ((s = light_tiers()) != WINGSPAN_OK) return s;
        HIP_TRY(hipStreamWaitEvent(c.st, side->join, 0));
    }

    if ((s = timer_start(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;
    s = launch_spill<V, true>(c, M, perm, B->ncols, nullptr, sink, c_col, c_val,
                              &stats.launches[WINGSPAN_TIER_SPILL]);
    if (s != WINGSPAN_OK) return s;
    if ((s = timer_stop(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;

    if (c.o.validate) {
        int32_t flags = 0;
        HIP_TRY(hipMemcpyAsync(&flags, &c.ctrl->error_flags, sizeof(int32_t), hipMemcpyDeviceToHost, c.st));
        HIP_TRY(hipStreamSynchronize(c.st));
        if (flags & (kErrRowMismatch | kErrProbeExhausted))
            return fail(WINGSPAN_ERR_INCONSISTENT, "C.row_ptr does not match the structure of A*B (flags %d)",
                        flags);
    }
    return WINGSPAN_OK;
}

// Single pass with sharded output: rows binned by products, each tier's
// numeric kernel claims a row's pool segment once the row's entry count is
// known and writes the sorted row there.
template <typename V>
wingspan_status sharded_impl(Ctx &c, const wingspan_csr *A, const wingspan_csr *B, int64_t *row_off,
                             int32_t *row_nnz, int32_t *pool_col, V *pool_val, int64_t cap, int64_t *used) {
    const int64_t m = A->nrows;
    // rows without products are written by the analysis (row_nnz = 0); their offsets here
    if (m > 0) {
        fill_i64<<<blocks_for(m, 256), 256, 0, c.st>>>(row_off, m, 0);
        LAUNCH_CHECK("fill offsets");
    }
    wingspan_status s = analyze(c, A, B, kModeSharded, nullptr, false, row_nnz);
    if (s != WINGSPAN_OK) return s;
    fill_stats(c, 2);
    wingspan_phase_stats &stats = g_stats[2];
    const Mats<V> M{A->row_ptr, A->col_idx, static_cast<const V *>(A->val),
                    B->row_ptr, B->col_idx, static_cast<const V *>(B->val)};
    const int32_t *perm = c.perm;
    RowSink sink;
    sink.claimed = &c.ctrl->pool_claimed;
    sink.row_off = row_off;
    sink.row_nnz = row_nnz;
    sink.cap = cap;

    if ((s = timer_start(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;
    for (int i = 0; i < kNumTiny; ++i) {
        const int b = kBinTiny0 + i;
        const int32_t cnt = c.host.bin_count[b];
        if (!cnt) continue;
        const int S = 8 << i;
        launch_tiny<V, true>(i, blocks_for(int64_t(cnt) * S, 256), c.st, M, perm + c.host.bin_offset[b], cnt,
                             nullptr, sink, pool_col, pool_val, c.ctrl);
        stats.launches[WINGSPAN_TIER_TINY]++;
    }
    LAUNCH_CHECK("tiny single pass");
    if ((s = timer_stop(c, WINGSPAN_TIER_TINY)) != WINGSPAN_OK) return s;

    if ((s = timer_start(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;
    for (int i = 0; i < kNumHash; ++i) {
        const int b = kBinHash0 + i;
        const int32_t cnt = c.host.bin_count[b];
        if (!cnt) continue;
        launch_hash<V, true>(kHashLog2Min + i, static_cast<unsigned>(cnt), c.st, M, perm + c.host.bin_offset[b],
                             B->ncols, nullptr, sink, pool_col, pool_val, c.ctrl);
        stats.launches[WINGSPAN_TIER_HASH]++;
    }
    LAUNCH_CHECK("hash single pass");
    if ((s = timer_stop(c, WINGSPAN_TIER_HASH)) != WINGSPAN_OK) return s;

    int32_t start, cnt;
    bin_range(c, kBinDense0, kNumClasses, &start, &cnt);
    if (cnt) {
        const int64_t entries = B->nrows * static_cast<int64_t>(c.L.nwin + 1);
        build_window_table<<<blocks_for(entries, 256), 256, 0, c.st>>>(B->row_ptr, B->col_idx, B->nrows, c.L.nwin,
                                                                       c.L.wcols, c.wtab);
        LAUNCH_CHECK("build_window_table");
    }
    if ((s = timer_start(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;
    if (cnt) {
        // binning sends dense rows here only in rank mode; the column bitmaps come from the kernel's own
        // structure pass
        rank_rows<<<blocks_for(cnt, 256), 256, 0, c.st>>>(perm + start, cnt, A->row_ptr, nullptr, nullptr,
                                                            c.rrows);
        LAUNCH_CHECK("rank rows");
        if (!c.o.wide_offsets && offsets_fit_32<V>(B))
            dense_rank_kernel<V, true, true><<<rank_grid(cnt), RankShape<V>::BLOCK, 0, c.st>>>(
                M, c.rrows, cnt, c.wtab, c.L.nwin, B->ncols, sink, pool_col, pool_val, c.ctrl, nullptr,
                c.L.row_words);
        else
            dense_rank_kernel<V, true, false><<<rank_grid(cnt), RankShape<V>::BLOCK, 0, c.st>>>(
                M, c.rrows, cnt, c.wtab, c.L.nwin, B->ncols, sink, pool_col, pool_val, c.ctrl, nullptr,
                c.L.row_words);
        stats.launches[WINGSPAN_TIER_DENSE]++;
        LAUNCH_CHECK("dense rank single pass");
    }
    if ((s = timer_stop(c, WINGSPAN_TIER_DENSE)) != WINGSPAN_OK) return s;

    if ((s = timer_start(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;
    s = launch_spill<V, true>(c, M, perm, B->ncols, nullptr, sink, pool_col, pool_val,
                              &stats.launches[WINGSPAN_TIER_SPILL]);
    if (s != WINGSPAN_OK) return s;
    if ((s = timer_stop(c, WINGSPAN_TIER_SPILL)) != WINGSPAN_OK) return s;

    HIP_TRY(hipMemcpyAsync(&c.host, c.ctrl, sizeof(Control), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if (c.host.error_flags & kErrProbeExhausted)
        return fail(WINGSPAN_ERR_INCONSISTENT, "a row's hash table filled up (flags %d)", c.host.error_flags);
    const int64_t total = static_cast<int64_t>(c.host.pool_claimed);
    *used = total;
    stats.c_nnz_total = total;
    if (total > cap)
        return fail(WINGSPAN_ERR_INSUFFICIENT_CAPACITY, "C has %lld entries but the pool holds %lld",
                    (long long)total, (long long)cap);
    return WINGSPAN_OK;
}

wingspan_status finish_timing(int phase) {
    if (!g_timer.on) return WINGSPAN_OK;
    for (int slot = 0; slot <= WINGSPAN_NUM_TIERS; ++slot) {
        HIP_TRY(hipEventSynchronize(g_timer.ev[2 * slot + 1]));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, g_timer.ev[2 * slot], g_timer.ev[2 * slot + 1]));
        if (slot == kSlotAnalysis) g_stats[phase].analysis_ms = ms;
        else g_stats[phase].kernel_ms[slot] = ms;
    }
    return WINGSPAN_OK;
}

wingspan_status setup(Ctx &c, const wingspan_csr *A, const wingspan_csr *B, const wingspan_options *opt,
                      void *ws, size_t ws_bytes, void *stream, size_t budget = 0) {
    wingspan_status s = parse_opts(opt, &c.o);
    if (s != WINGSPAN_OK) return s;
    c.L = plan(A, B, c.o, budget);
    if (ws_bytes < c.L.total)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", ws_bytes, c.L.total);
    if (!ws) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kAlign);
    c.st = static_cast<hipStream_t>(stream);
    carve(c, ws);
    if (!c.o.dense_min_explicit && c.L.cache_rows > 0) c.o.dense_min_nnz = kCachedDenseMin;
    return WINGSPAN_OK;
}

// ---------------------------------------------------------------------------
// Elementwise operations (SpAdd, Hadamard): workspace layout and checks.
// ---------------------------------------------------------------------------
// The tiling an elementwise structure call leaves in its workspace (tile
// boundaries and each tile's first place in C), remembered on the host so a
// values call with the same operation, patterns and workspace skips
// recomputing it. Every call of this library that is handed a workspace
// forgets the plans kept in the memory it covers.
struct EwPlanKey {
    const char *ws;
    size_t bytes;
    int op;
    int64_t m, n, a_nnz, b_nnz;
    const int32_t *a_rp, *a_col, *b_rp, *b_col;
    bool same(const EwPlanKey &o) const {
        return ws == o.ws && op == o.op && m == o.m && n == o.n && a_nnz == o.a_nnz && b_nnz == o.b_nnz &&
               a_rp == o.a_rp && a_col == o.a_col && b_rp == o.b_rp && b_col == o.b_col;
    }
    bool overlaps(const char *lo, size_t len) const { return ws < lo + len && lo < ws + bytes; }
};

std::mutex g_ew_mu;
std::vector<EwPlanKey> g_ew_plans;
constexpr size_t kEwMaxPlans = 16;

EwPlanKey ew_key_of(int op, const wingspan_csr *A, const wingspan_csr *B, void *ws, size_t bytes) {
    return EwPlanKey{static_cast<const char *>(ws), bytes, op, A->nrows, A->ncols, A->nnz, B->nnz,
                     A->row_ptr, A->col_idx, B->row_ptr, B->col_idx};
}

void ew_forget(const void *ws, size_t bytes) {
    if (!ws) return;
    const char *lo = static_cast<const char *>(ws);
    std::lock_guard<std::mutex> lk(g_ew_mu);
    g_ew_plans.erase(std::remove_if(g_ew_plans.begin(), g_ew_plans.end(),
                                    [&](const EwPlanKey &k) { return k.overlaps(lo, bytes); }),
                     g_ew_plans.end());
}

bool ew_known(const EwPlanKey &key) {
    std::lock_guard<std::mutex> lk(g_ew_mu);
    for (const EwPlanKey &k : g_ew_plans)
        if (k.same(key)) return true;
    return false;
}

void ew_remember(const EwPlanKey &key) {
    std::lock_guard<std::mutex> lk(g_ew_mu);
    g_ew_plans.erase(std::remove_if(g_ew_plans.begin(), g_ew_plans.end(),
                                    [&](const EwPlanKey &k) { return k.overlaps(key.ws, key.bytes); }),
                     g_ew_plans.end());
    if (g_ew_plans.size() >= kEwMaxPlans) g_ew_plans.erase(g_ew_plans.begin());
    g_ew_plans.push_back(key);
}

struct EwLayout {
    size_t off_dups, off_split_a, off_split_b, off_split_r, off_tile_cnt, off_tile_off, off_partials, total;
    int64_t ntiles;
};

// The merged sequence's tiles (kEwTile entries of A and B together).
int64_t ew_tiles(const wingspan_csr *A, const wingspan_csr *B) { return (A->nnz + B->nnz + kEwTile - 1) / kEwTile; }

EwLayout ew_plan(const wingspan_csr *A, const wingspan_csr *B) {
    EwLayout L{};
    const int64_t m = std::max<int64_t>(A->nrows, 1);
    L.ntiles = ew_tiles(A, B);
    const int64_t nb = L.ntiles + 1;   // boundaries
    size_t off = 0;
    L.off_dups = off;
    off += align_up(sizeof(int32_t) * m);
    L.off_split_a = off;
    off += align_up(sizeof(int64_t) * nb);
    L.off_split_b = off;
    off += align_up(sizeof(int64_t) * nb);
    L.off_split_r = off;
    off += align_up(sizeof(int32_t) * nb);
    L.off_tile_cnt = off;
    off += align_up(sizeof(int32_t) * nb);
    L.off_tile_off = off;
    off += align_up(sizeof(int64_t) * (nb + 1));
    L.off_partials = off;
    const int64_t n = std::max<int64_t>(m + 1, nb);
    off += align_up(sizeof(int64_t) * ((n + kScanTile - 1) / kScanTile + 2));
    L.total = off;
    return L;
}

wingspan_status ew_check(int op, const wingspan_csr *A, const wingspan_csr *B) {
    if (op != WINGSPAN_OP_ADD && op != WINGSPAN_OP_HADAMARD)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "op must be WINGSPAN_OP_ADD or WINGSPAN_OP_HADAMARD");
    wingspan_status s = check_csr_desc(A, "A");
    if (s != WINGSPAN_OK) return s;
    if ((s = check_csr_desc(B, "B")) != WINGSPAN_OK) return s;
    if (A->nrows != B->nrows || A->ncols != B->ncols)
        return fail(WINGSPAN_ERR_DIMENSION_MISMATCH, "A is %lldx%lld but B is %lldx%lld", (long long)A->nrows,
                    (long long)A->ncols, (long long)B->nrows, (long long)B->ncols);
    return WINGSPAN_OK;
}

wingspan_status ew_workspace(const wingspan_csr *A, const wingspan_csr *B, void *ws, size_t ws_bytes,
                             EwLayout *L) {
    *L = ew_plan(A, B);
    if (ws_bytes < L->total)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", ws_bytes, L->total);
    if (!ws) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kAlign);
    return WINGSPAN_OK;
}

struct EwTiles {
    int64_t *split_a, *split_b, *tile_off;
    int32_t *split_r, *tile_cnt, *dups;
};

EwTiles ew_arrays(Ctx &c, const EwLayout &L) {
    EwTiles T;
    T.split_a = reinterpret_cast<int64_t *>(c.ws + L.off_split_a);
    T.split_b = reinterpret_cast<int64_t *>(c.ws + L.off_split_b);
    T.split_r = reinterpret_cast<int32_t *>(c.ws + L.off_split_r);
    T.tile_cnt = reinterpret_cast<int32_t *>(c.ws + L.off_tile_cnt);
    T.tile_off = reinterpret_cast<int64_t *>(c.ws + L.off_tile_off);
    T.dups = reinterpret_cast<int32_t *>(c.ws + L.off_dups);
    c.partials = reinterpret_cast<int64_t *>(c.ws + L.off_partials);
    return T;
}

// The tiles' boundaries, then their counts (with PER_ROW also each row's
// common coordinates, into T.dups, which the caller zeroed). nrows >= 1 and
// ntiles >= 1.
template <bool PER_ROW>
wingspan_status ew_count_tiles(Ctx &c, int op, const wingspan_csr *A, const wingspan_csr *B, const EwLayout &L,
                               const EwTiles &T) {
    const int m = static_cast<int>(A->nrows);
    ew_tile_splits<<<blocks_for((L.ntiles + 1) * kWave, 256), 256, 0, c.st>>>(
        A->row_ptr, A->col_idx, B->row_ptr, B->col_idx, m, L.ntiles, T.split_a, T.split_b, T.split_r);
    LAUNCH_CHECK("elementwise splits");
    ew_tile_count<PER_ROW><<<static_cast<unsigned>(L.ntiles), kEwBlock, 0, c.st>>>(
        A->row_ptr, A->col_idx, B->row_ptr, B->col_idx, T.split_a, T.split_b, T.split_r, op, T.tile_cnt, T.dups);
    LAUNCH_CHECK("elementwise count");
    return WINGSPAN_OK;
}

// Each tile's first place in C, from the tile counts.
wingspan_status ew_scan_tiles(Ctx &c, const EwLayout &L, const EwTiles &T) {
    // one workgroup scans a few thousand tile counts, the tiled scan more (measured: 25 us for 16 K counts in
    // one workgroup)
    if (L.ntiles <= 2048) {
        scan_one_block<EwTileIn><<<1, 1024, 0, c.st>>>(EwTileIn{T.tile_cnt}, L.ntiles, T.tile_off);
        LAUNCH_CHECK("elementwise tile scan");
        return WINGSPAN_OK;
    }
    return run_scan(c, EwTileIn{T.tile_cnt}, L.ntiles, T.tile_off);
}

// The values; `planned`: the workspace holds this problem's tiling from an earlier call.
template <typename V>
wingspan_status ew_values_impl(Ctx &c, int op, const wingspan_csr *A, const wingspan_csr *B, const EwLayout &L,
                               int32_t *c_col, V *c_val, bool planned) {
    if (A->nrows == 0 || L.ntiles == 0) return WINGSPAN_OK;
    if (op == WINGSPAN_OP_HADAMARD && (A->nnz == 0 || B->nnz == 0)) return WINGSPAN_OK;   // C is empty
    const EwTiles T = ew_arrays(c, L);
    wingspan_status s;
    if (!planned) {
        if ((s = ew_count_tiles<false>(c, op, A, B, L, T)) != WINGSPAN_OK) return s;
        if ((s = ew_scan_tiles(c, L, T)) != WINGSPAN_OK) return s;
    }
    const V *av = static_cast<const V *>(A->val), *bv = static_cast<const V *>(B->val);
    const unsigned grid = static_cast<unsigned>(L.ntiles);
    if (op == WINGSPAN_OP_ADD)
        ew_tile_write<V, kEwAdd><<<grid, kEwBlock, 0, c.st>>>(A->row_ptr, A->col_idx, av, B->row_ptr, B->col_idx, bv,
                                                              T.split_a, T.split_b, T.split_r, T.tile_off, c_col,
                                                              c_val);
    else
        ew_tile_write<V, kEwMul><<<grid, kEwBlock, 0, c.st>>>(A->row_ptr, A->col_idx, av, B->row_ptr, B->col_idx, bv,
                                                              T.split_a, T.split_b, T.split_r, T.tile_off, c_col,
                                                              c_val);
    LAUNCH_CHECK("elementwise write");
    return WINGSPAN_OK;
}

// ---------------------------------------------------------------------------
// SpMSpV: workspace layout and checks.
// ---------------------------------------------------------------------------
constexpr int64_t kSvMaxGrid = 8192;   // scatter workgroups at most (grid-stride beyond)

constexpr int64_t kSvMaxTable = int64_t(1) << 25;   // (range, chunk) counts of the bucketed scatter at most
constexpr int64_t kSvBucketGrid = 512;              // its workgroups at most (grid-stride beyond)

struct SvLayout {
    size_t off_pref, off_partials, off_flag, off_yval, off_tiles, off_tile_pre, off_err, total;
    size_t off_tab, off_gpos, off_piece_pre, off_tmp_row, off_tmp_val, off_srt_row, off_srt_val;
    int64_t ntiles;
    int64_t nchunks;   // binning chunks (bounded by At's entries)
    bool bucketed;     // the bucketed scatter (else the atomic one)
};

SvLayout sv_plan(const wingspan_csr *At, int64_t nnz_x) {
    SvLayout L{};
    const int64_t m = std::max<int64_t>(At->ncols, 1), nx = std::max<int64_t>(nnz_x, 0);
    L.ntiles = (m + kSvTile - 1) / kSvTile;
    size_t off = 0;
    // first the tiles' prefix, its total (y's entry count) last, then the error word: the total and the error
    // word are read back in one copy. (Measured: the scatter runs about 20% slower with these small arrays
    // placed just past the map's accumulators.)
    L.off_tile_pre = off;
    L.off_err = off + sizeof(int64_t) * (L.ntiles + 1);
    off += align_up(sizeof(int64_t) * (L.ntiles + 1) + sizeof(int64_t));
    L.off_tiles = off;
    off += align_up(sizeof(int32_t) * L.ntiles);
    L.off_pref = off;
    off += align_up(sizeof(int64_t) * (nx + 1));
    // the bucketed scatter: ranges of y are the emission tiles; its buffers are sized by At's entries (the
    // product count is known on the device only)
    const int64_t nnz = std::max<int64_t>(At->nnz, 1);
    L.nchunks = (nnz + kSvBin - 1) / kSvBin;
    L.bucketed = L.ntiles <= kSvMaxRanges && L.ntiles * L.nchunks <= kSvMaxTable;
    const int64_t ntab = L.bucketed ? L.ntiles * L.nchunks : 0;
    L.off_partials = off;
    off += align_up(sizeof(int64_t) * ((std::max<int64_t>(nx, ntab) + kScanTile - 1) / kScanTile + 2));
    L.off_flag = off;
    off += align_up(static_cast<size_t>((m + 3) / 4) * 4);   // cleared as int32 words
    L.off_yval = off;
    off += align_up(sizeof(double) * m);
    if (L.bucketed) {
        L.off_tab = off;
        off += align_up(sizeof(int32_t) * ntab);
        L.off_gpos = off;
        off += align_up(sizeof(int64_t) * (ntab + 1));
        L.off_piece_pre = off;
        off += align_up(sizeof(int64_t) * (L.ntiles + 1));
        L.off_tmp_row = off;
        off += align_up(sizeof(int32_t) * nnz);
        L.off_tmp_val = off;
        off += align_up(sizeof(double) * nnz);
        L.off_srt_row = off;
        off += align_up(sizeof(int32_t) * nnz);
        L.off_srt_val = off;
        off += align_up(sizeof(double) * nnz);
    }
    L.total = off;
    return L;
}

wingspan_status sv_check(const wingspan_csr *At, int64_t nnz_x) {
    wingspan_status s = check_csr_desc(At, "At");
    if (s != WINGSPAN_OK) return s;
    if (nnz_x < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "nnz_x is negative");
    if (nnz_x > At->nrows)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "x has %lld entries but length %lld", (long long)nnz_x,
                    (long long)At->nrows);
    return WINGSPAN_OK;
}

template <typename V>
wingspan_status sv_impl(Ctx &c, const wingspan_csr *At, const SvLayout &L, const int32_t *x_idx, const V *x_val,
                        int64_t nnz_x, int32_t *y_idx, V *y_val, int64_t y_cap, int64_t *y_nnz) {
    const int64_t m = At->ncols, n = At->nrows;
    int32_t *err = reinterpret_cast<int32_t *>(c.ws + L.off_err);
    int64_t *pref = reinterpret_cast<int64_t *>(c.ws + L.off_pref);
    uint8_t *flag = reinterpret_cast<uint8_t *>(c.ws + L.off_flag);
    double *yval = reinterpret_cast<double *>(c.ws + L.off_yval);
    int32_t *tiles = reinterpret_cast<int32_t *>(c.ws + L.off_tiles);
    int64_t *tile_pre = reinterpret_cast<int64_t *>(c.ws + L.off_tile_pre);
    *y_nnz = 0;
    if (m == 0) return WINGSPAN_OK;
    // an empty map; x's columns' lengths scanned (checking x on the way); the scatter, sized by At's entries
    // and reading the product count on the device
    const int64_t nwords = (m + 3) / 4;
    sv_clear<<<blocks_for(std::max<int64_t>(nwords, m), 256), 256, 0, c.st>>>(
        reinterpret_cast<int32_t *>(flag), nwords, reinterpret_cast<int64_t *>(yval), m, err);
    LAUNCH_CHECK("spmspv clear");
    if (nnz_x > 0) {
        // (the tiled scan: one workgroup walking x would wait on each entry's two dependent loads in turn)
        c.partials = reinterpret_cast<int64_t *>(c.ws + L.off_partials);
        wingspan_status s = run_scan(c, SvLenIn{At->row_ptr, x_idx, n, err}, nnz_x, pref);
        if (s != WINGSPAN_OK) return s;
        if (At->nnz > 0 && L.bucketed) {
            // products sorted by range of y, then each range summed in LDS (grids sized by At's entries; the
            // kernels read the product count on the device)
            const int nr = static_cast<int>(L.ntiles);
            const int64_t nc = L.nchunks;
            int32_t *tab = reinterpret_cast<int32_t *>(c.ws + L.off_tab);
            int64_t *gpos = reinterpret_cast<int64_t *>(c.ws + L.off_gpos);
            int32_t *tmp_row = reinterpret_cast<int32_t *>(c.ws + L.off_tmp_row);
            double *tmp_val = reinterpret_cast<double *>(c.ws + L.off_tmp_val);
            int32_t *srt_row = reinterpret_cast<int32_t *>(c.ws + L.off_srt_row);
            double *srt_val = reinterpret_cast<double *>(c.ws + L.off_srt_val);
            const unsigned grid = static_cast<unsigned>(std::min<int64_t>(nc, kSvBucketGrid));
            sv_bin<V><<<grid, kSvBinBlock, 0, c.st>>>(At->row_ptr, At->col_idx, static_cast<const V *>(At->val),
                                                      x_idx, x_val, static_cast<int>(nnz_x), pref, err, nr, nc, tab,
                                                      tmp_row, tmp_val);
            LAUNCH_CHECK("spmspv bin");
            if ((s = run_scan(c, SvTabIn{tab, pref, static_cast<int>(nnz_x), nc}, nr * nc, gpos)) != WINGSPAN_OK)
                return s;
            sv_place<<<grid, kSvBinBlock, 0, c.st>>>(tmp_row, tmp_val, pref, static_cast<int>(nnz_x), err, nr, nc,
                                                     tab, gpos, srt_row, srt_val);
            int64_t *piece_pre = reinterpret_cast<int64_t *>(c.ws + L.off_piece_pre);
            scan_one_block<SvPiecesIn><<<1, 1024, 0, c.st>>>(SvPiecesIn{gpos, nc}, nr, piece_pre);
            const int64_t pieces = nr + (At->nnz + kSvPieceMax - 1) / kSvPieceMax;   // at most
            sv_accumulate<<<static_cast<unsigned>(std::min<int64_t>(pieces, kSvBucketGrid)), kSvAccBlock, 0, c.st>>>(
                srt_row, srt_val, err, nr, nc, gpos, piece_pre, flag, yval);
            LAUNCH_CHECK("spmspv accumulate");
        } else if (At->nnz > 0) {
            const int64_t chunks = (At->nnz + kSvChunk - 1) / kSvChunk;
            sv_scatter<V><<<static_cast<unsigned>(std::min<int64_t>(chunks, kSvMaxGrid)), kSvBlock, 0, c.st>>>(
                At->row_ptr, At->col_idx, static_cast<const V *>(At->val), x_idx, x_val, static_cast<int>(nnz_x),
                pref, err, flag, yval);
            LAUNCH_CHECK("spmspv scatter");
        }
    }
    // coalesce the map tile by tile: counts, their scan (the total lands next to the error word), then y
    const unsigned nt = static_cast<unsigned>(L.ntiles);
    sv_tile_count<<<nt, kSvTileBlock, 0, c.st>>>(reinterpret_cast<const uint32_t *>(flag), m, tiles);
    scan_one_block<SvTileIn><<<1, 1024, 0, c.st>>>(SvTileIn{tiles}, L.ntiles, tile_pre);
    sv_emit_tiles<V><<<nt, kSvTileBlock, 0, c.st>>>(flag, yval, tile_pre, m, y_cap, y_idx, y_val);
    LAUNCH_CHECK("spmspv emit");
    struct {
        int64_t total;
        int32_t err;
        int32_t pad;
    } back{};
    static_assert(sizeof(back) == 16, "total then error word");
    HIP_TRY(hipMemcpyAsync(&back, tile_pre + L.ntiles, sizeof(back), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if (back.err) return fail(WINGSPAN_ERR_INVALID_MATRIX, "x's indices are not strictly increasing in [0, %lld)",
                              (long long)n);
    *y_nnz = back.total;
    if (back.total > y_cap)
        return fail(WINGSPAN_ERR_INSUFFICIENT_CAPACITY, "y has %lld entries but y_cap is %lld",
                    (long long)back.total, (long long)y_cap);
    return WINGSPAN_OK;
}

// ---------------------------------------------------------------------------
// Outer-product SpGEMM: workspace layout and checks. The count's arrays come
// first, at offsets that do not depend on the product count P.
// ---------------------------------------------------------------------------
constexpr int64_t kOpLongGrid = 2048;   // coalesce workgroups for long rows at most (grid-stride beyond)
constexpr int64_t kOpHugeGrid = 512;    // the same for rows past kOpRowCap (one or two workgroups per CU)

struct OpLayout {
    size_t off_ctr, off_pref, off_partials, off_part_key, off_part_val, off_part_len, off_row_cnt, off_row_fill,
        off_bucket, off_row_nnz, off_long, off_bkt_col, off_bkt_val, off_out_val, total;
};

OpLayout op_plan(const wingspan_csr *At, const wingspan_csr *B, int64_t P) {
    OpLayout L{};
    const int64_t K = std::max<int64_t>(At->nrows, 1), m = std::max<int64_t>(At->ncols, 1);
    const int64_t p = std::max<int64_t>(P, 1), chunks = (p + kOpChunk - 1) / kOpChunk;
    size_t off = 0;
    L.off_ctr = off;
    off += align_up(sizeof(int32_t) * 4);
    L.off_pref = off;
    off += align_up(sizeof(int64_t) * (K + 1));
    L.off_partials = off;
    const int64_t n = std::max<int64_t>(K, m) + 1;
    off += align_up(sizeof(int64_t) * ((n + kScanTile - 1) / kScanTile + 2));
    L.off_part_key = off;   // after the bucket step: two int32 column arrays of p for the long-row merge
    off += align_up(sizeof(int64_t) * p);
    L.off_part_val = off;
    off += align_up(sizeof(double) * p);
    L.off_part_len = off;
    off += align_up(sizeof(int32_t) * chunks);
    L.off_row_cnt = off;
    off += align_up(sizeof(int32_t) * m);
    L.off_row_fill = off;
    off += align_up(sizeof(int32_t) * m);
    L.off_bucket = off;
    off += align_up(sizeof(int64_t) * (m + 1));
    L.off_row_nnz = off;
    off += align_up(sizeof(int32_t) * m);
    L.off_long = off;
    off += align_up(sizeof(int32_t) * m);
    L.off_bkt_col = off;
    off += align_up(sizeof(int32_t) * p);
    L.off_bkt_val = off;
    off += align_up(sizeof(double) * p);
    L.off_out_val = off;
    off += align_up(sizeof(double) * p);
    L.total = off;
    (void)B;
    return L;
}

wingspan_status op_check(const wingspan_csr *At, const wingspan_csr *B) {
    wingspan_status s = check_csr_desc(At, "At");
    if (s != WINGSPAN_OK) return s;
    if ((s = check_csr_desc(B, "B")) != WINGSPAN_OK) return s;
    if (At->nrows != B->nrows)
        return fail(WINGSPAN_ERR_DIMENSION_MISMATCH, "At has %lld rows (A's columns) but B has %lld rows",
                    (long long)At->nrows, (long long)B->nrows);
    return WINGSPAN_OK;
}

wingspan_status op_workspace_ok(void *ws, size_t bytes, size_t need) {
    if (bytes < need) return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", bytes, need);
    if (!ws) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kAlign);
    return WINGSPAN_OK;
}

// The per-k product prefix into pref and its total, read back.
wingspan_status op_count(Ctx &c, const wingspan_csr *At, const wingspan_csr *B, const OpLayout &L, int64_t *P) {
    int64_t *pref = reinterpret_cast<int64_t *>(c.ws + L.off_pref);
    c.partials = reinterpret_cast<int64_t *>(c.ws + L.off_partials);
    *P = 0;
    if (At->nrows == 0) return WINGSPAN_OK;
    wingspan_status s = run_scan(c, OpProdIn{At->row_ptr, B->row_ptr}, At->nrows, pref);
    if (s != WINGSPAN_OK) return s;
    HIP_TRY(hipMemcpyAsync(P, pref + At->nrows, sizeof(int64_t), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    return WINGSPAN_OK;
}

template <typename V>
wingspan_status op_impl(Ctx &c, const wingspan_csr *At, const wingspan_csr *B, const OpLayout &L, int64_t P,
                        int64_t *c_rp, int32_t *c_col, V *c_val, int64_t c_cap, int64_t *c_nnz) {
    const int64_t K = At->nrows, m = At->ncols;
    auto at = [&](size_t off) { return c.ws + off; };
    int32_t *ctr = reinterpret_cast<int32_t *>(at(L.off_ctr));
    const int64_t *pref = reinterpret_cast<const int64_t *>(at(L.off_pref));
    int64_t *part_key = reinterpret_cast<int64_t *>(at(L.off_part_key));
    double *part_val = reinterpret_cast<double *>(at(L.off_part_val));
    int32_t *part_len = reinterpret_cast<int32_t *>(at(L.off_part_len));
    int32_t *row_cnt = reinterpret_cast<int32_t *>(at(L.off_row_cnt));
    int32_t *row_fill = reinterpret_cast<int32_t *>(at(L.off_row_fill));
    int64_t *bucket = reinterpret_cast<int64_t *>(at(L.off_bucket));
    int32_t *row_nnz = reinterpret_cast<int32_t *>(at(L.off_row_nnz));
    int32_t *long_rows = reinterpret_cast<int32_t *>(at(L.off_long));
    int32_t *bkt_col = reinterpret_cast<int32_t *>(at(L.off_bkt_col));
    double *bkt_val = reinterpret_cast<double *>(at(L.off_bkt_val));
    V *out_val = reinterpret_cast<V *>(at(L.off_out_val));
    *c_nnz = 0;
    if (m == 0) {
        // C has no rows: its row pointer is the single 0
        fill_i64<<<1, 64, 0, c.st>>>(c_rp, 1, 0);
        LAUNCH_CHECK("outer empty");
        return WINGSPAN_OK;
    }
    fill_i32<<<1, 64, 0, c.st>>>(ctr, 4, 0);
    fill_i32<<<blocks_for(m, 256), 256, 0, c.st>>>(row_cnt, m, 0);
    fill_i32<<<blocks_for(m, 256), 256, 0, c.st>>>(row_fill, m, 0);
    LAUNCH_CHECK("outer clear");
    const int64_t chunks = (P + kOpChunk - 1) / kOpChunk;
    // 1. the workgroups' partial Cs
    if (P > 0) {
        op_expand<V><<<static_cast<unsigned>(chunks), kOpBlock, 0, c.st>>>(
            At->row_ptr, At->col_idx, static_cast<const V *>(At->val), B->row_ptr, B->col_idx,
            static_cast<const V *>(B->val), static_cast<int>(K), pref, P, part_key, part_val, part_len, row_cnt);
        LAUNCH_CHECK("outer expand");
    }
    // 2. coalesce: row buckets, then each bucket sorted and compacted
    wingspan_status s = run_scan(c, CountIn{row_cnt}, m, bucket);
    if (s != WINGSPAN_OK) return s;
    if (P > 0) {
        op_bucket<<<static_cast<unsigned>(chunks), 256, 0, c.st>>>(part_key, part_val, part_len, bucket, row_fill,
                                                                   bkt_col, bkt_val);
        LAUNCH_CHECK("outer bucket");
    }
    op_merge_short<32, V><<<blocks_for(m, 256 / 32), 256, 0, c.st>>>(bucket, m, bkt_col, bkt_val, out_val, row_nnz,
                                                                      long_rows, ctr);
    op_merge_short<64, V><<<blocks_for(m, 256 / 64), 256, 0, c.st>>>(bucket, m, bkt_col, bkt_val, out_val, row_nnz,
                                                                      long_rows, ctr);
    op_merge_long<V><<<static_cast<unsigned>(std::min<int64_t>(m, kOpLongGrid)), kOpRowBlock, 0, c.st>>>(
        bucket, bkt_col, bkt_val, out_val, row_nnz, long_rows, ctr);
    // rows past kOpRowCap: the partial Cs are no longer needed, so their arrays
    // hold the sorted runs (X: columns in part_key's first half, values in
    // part_val; Y: columns in its second half, values in bkt_val)
    int32_t *run_col = reinterpret_cast<int32_t *>(part_key);
    op_merge_huge<V><<<static_cast<unsigned>(std::min<int64_t>(m, kOpHugeGrid)), kOpHugeBlock, 0, c.st>>>(
        bucket, m, bkt_col, bkt_val, out_val, row_nnz, long_rows, ctr, run_col, part_val,
        run_col + std::max<int64_t>(P, 1));
    LAUNCH_CHECK("outer merge");
    // 3. C.row_ptr, then the rows gathered into CSR
    if ((s = run_scan(c, CountIn{row_nnz}, m, c_rp)) != WINGSPAN_OK) return s;
    HIP_TRY(hipMemcpyAsync(c_nnz, c_rp + m, sizeof(int64_t), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    if (*c_nnz > c_cap)
        return fail(WINGSPAN_ERR_INSUFFICIENT_CAPACITY, "C has %lld entries but c_capacity is %lld",
                    (long long)*c_nnz, (long long)c_cap);
    if (*c_nnz > 0) {
        gather_rows<V><<<static_cast<unsigned>((*c_nnz + kGatherChunk - 1) / kGatherChunk), 256, 0, c.st>>>(
            m, bucket, c_rp, bkt_col, out_val, c_col, c_val);
        LAUNCH_CHECK("outer gather");
    }
    return WINGSPAN_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Static scratch of wingspan_spgemm_noalloc: a device array in the library's
// code object, so that entry point needs no allocation. Every device the
// library runs on holds its own copy, at its own address, until the process
// ends. Host code never uses the array's name as an address (on the host it
// names a stand-in, not device memory): it takes the device address from
// hipGetSymbolAddress, once per device, with that device current.
// ---------------------------------------------------------------------------
static __device__ __align__(256) char wsp_static_scratch[WINGSPAN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of the static scratch.
wingspan_status static_scratch(void **out) {
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(WINGSPAN_ERR_UNSUPPORTED, "device %d: the static scratch is kept for devices 0..%d", dev,
                    kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(wsp_static_scratch)));
        if (p == nullptr || reinterpret_cast<uintptr_t>(p) % kAlign != 0)
            return fail(WINGSPAN_ERR_HIP, "hipGetSymbolAddress gave an unusable scratch address %p", p);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return WINGSPAN_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

int wingspan_abi_version(void) { return WINGSPAN_ABI_VERSION; }

const char *wingspan_last_error(void) { return g_err.c_str(); }

wingspan_status wingspan_last_stats(int phase, wingspan_phase_stats *out) {
    if (phase < 0 || phase > 2 || !out) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bad phase or NULL out");
    *out = g_stats[phase];
    return WINGSPAN_OK;
}

wingspan_status wingspan_spgemm_workspace_size(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                               const wingspan_options *options, size_t *bytes) {
    g_err.clear();
    if (!bytes) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bytes is NULL");
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    Opts o;
    if ((s = parse_opts(options, &o)) != WINGSPAN_OK) return s;
    *bytes = plan(A, B, o).total;
    return WINGSPAN_OK;
}

static wingspan_status symbolic_entry(const wingspan_csr *A, const wingspan_csr *B, int64_t *c_row_ptr_dev,
                                      int64_t *c_nnz, void *workspace_dev, size_t workspace_bytes, void *stream,
                                      const wingspan_options *options, Ctx &c, size_t budget = 0) {
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if (!c_nnz) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_nnz is NULL");
    if ((s = setup(c, A, B, options, workspace_dev, workspace_bytes, stream, budget)) != WINGSPAN_OK) return s;
    if ((s = timer_begin(c.o.timing)) != WINGSPAN_OK) return s;
    if ((s = symbolic_impl(c, A, B, c_row_ptr_dev, c_nnz)) != WINGSPAN_OK) return s;
    return finish_timing(0);
}

wingspan_status wingspan_spgemm_symbolic(const wingspan_csr *A, const wingspan_csr *B, int64_t *c_row_ptr_dev,
                                         int64_t *c_nnz, void *workspace_dev, size_t workspace_bytes,
                                         void *stream, const wingspan_options *options) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    Ctx c{};
    return symbolic_entry(A, B, c_row_ptr_dev, c_nnz, workspace_dev, workspace_bytes, stream, options, c);
}

static wingspan_status numeric_entry(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                     const int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                     void *workspace_dev, size_t workspace_bytes, void *stream,
                                     const wingspan_options *options, bool have_pref, Ctx &c) {
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if (!have_pref && (s = setup(c, A, B, options, workspace_dev, workspace_bytes, stream)) != WINGSPAN_OK)
        return s;
    if ((s = timer_begin(c.o.timing)) != WINGSPAN_OK) return s;
    c.dtype_f64 = dtype == WINGSPAN_F64 ? 1 : 0;
    if (dtype == WINGSPAN_F32)
        s = numeric_impl<float>(c, A, B, c_row_ptr_dev, c_col_idx_dev, static_cast<float *>(c_val_dev), have_pref);
    else
        s = numeric_impl<double>(c, A, B, c_row_ptr_dev, c_col_idx_dev, static_cast<double *>(c_val_dev),
                                 have_pref);
    if (s != WINGSPAN_OK) return s;
    return finish_timing(1);
}

wingspan_status wingspan_spgemm_numeric(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                        const int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                        void *workspace_dev, size_t workspace_bytes, void *stream,
                                        const wingspan_options *options) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    Ctx c{};
    return numeric_entry(A, B, dtype, c_row_ptr_dev, c_col_idx_dev, c_val_dev, workspace_dev, workspace_bytes,
                         stream, options, false, c);
}

wingspan_status wingspan_spgemm(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                int64_t c_capacity, int64_t *c_nnz, void *workspace_dev, size_t workspace_bytes,
                                void *stream, const wingspan_options *options) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (c_capacity < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_capacity is negative");
    Ctx c{};
    wingspan_status s =
        symbolic_entry(A, B, c_row_ptr_dev, c_nnz, workspace_dev, workspace_bytes, stream, options, c);
    if (s != WINGSPAN_OK) return s;
    if (*c_nnz > c_capacity)
        return fail(WINGSPAN_ERR_INSUFFICIENT_CAPACITY, "nnz(C) = %lld exceeds c_capacity = %lld",
                    (long long)*c_nnz, (long long)c_capacity);
    if (*c_nnz > 0 && (!c_col_idx_dev || !c_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_col_idx_dev or c_val_dev is NULL");
    return numeric_entry(A, B, dtype, c_row_ptr_dev, c_col_idx_dev, c_val_dev, workspace_dev, workspace_bytes,
                         stream, options, true, c);
}

wingspan_status wingspan_spgemm_noalloc(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                        int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                        int64_t c_capacity, int64_t *c_nnz, void *stream,
                                        const wingspan_options *options) {
    g_err.clear();
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (c_capacity < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_capacity is negative");
    if (!c_nnz) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_nnz is NULL");
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    Opts o;
    if ((s = parse_opts(options, &o)) != WINGSPAN_OK) return s;
    if (o.timing)   // the timing events would be created (allocated) on first use
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "options->timing is not available without allocation");
    const size_t cap = WINGSPAN_NOALLOC_SCRATCH_BYTES;
    const size_t need = plan(A, B, o, cap).total;
    if (need > cap)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL,
                    "this product needs %zu bytes of scratch; the static scratch holds %zu", need, cap);
    void *scratch = nullptr;
    if ((s = static_scratch(&scratch)) != WINGSPAN_OK) return s;
    Ctx c{};
    c.side_ok = false;   // a side stream and its events would be created on first use
    s = symbolic_entry(A, B, c_row_ptr_dev, c_nnz, scratch, cap, stream, options, c, cap);
    if (s != WINGSPAN_OK) return s;
    if (*c_nnz > c_capacity)
        return fail(WINGSPAN_ERR_INSUFFICIENT_CAPACITY, "nnz(C) = %lld exceeds c_capacity = %lld",
                    (long long)*c_nnz, (long long)c_capacity);
    if (*c_nnz > 0 && (!c_col_idx_dev || !c_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_col_idx_dev or c_val_dev is NULL");
    return numeric_entry(A, B, dtype, c_row_ptr_dev, c_col_idx_dev, c_val_dev, scratch, cap, stream, options, true,
                         c);
}

wingspan_status wingspan_spgemm_row_products(const wingspan_csr *A, const wingspan_csr *B,
                                             int64_t *row_products_dev, void *workspace_dev, size_t workspace_bytes,
                                             void *stream) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    if (A->nrows > 0 && !row_products_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "row_products_dev is NULL");
    Ctx c{};
    if ((s = setup(c, A, B, nullptr, workspace_dev, workspace_bytes, stream)) != WINGSPAN_OK) return s;
    if (A->nrows == 0) return WINGSPAN_OK;
    // the analysis pass of both phases: B-row lengths scanned over A's entries, then per-row differences
    if ((s = run_scan(c, BRowLenIn{A->col_idx, B->row_ptr}, A->nnz, c.pref)) != WINGSPAN_OK) return s;
    row_products_kernel<<<blocks_for(A->nrows, 256), 256, 0, c.st>>>(A->row_ptr, c.pref, A->nrows, row_products_dev);
    LAUNCH_CHECK("row products");
    return WINGSPAN_OK;
}

wingspan_status wingspan_spgemm_sharded(const wingspan_csr *A, const wingspan_csr *B, wingspan_dtype dtype,
                                        int64_t *row_off_dev, int32_t *row_nnz_dev, int32_t *pool_col_dev,
                                        void *pool_val_dev, int64_t pool_capacity, int64_t *pool_used,
                                        void *workspace_dev, size_t workspace_bytes, void *stream,
                                        const wingspan_options *options) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    wingspan_status s = check_pair(A, B);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!pool_used) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "pool_used is NULL");
    if (pool_capacity < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "pool_capacity is negative");
    if (A->nrows > 0 && (!row_off_dev || !row_nnz_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "row_off_dev or row_nnz_dev is NULL");
    if (pool_capacity > 0 && (!pool_col_dev || !pool_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "pool_col_dev or pool_val_dev is NULL");
    Ctx c{};
    if ((s = setup(c, A, B, options, workspace_dev, workspace_bytes, stream)) != WINGSPAN_OK) return s;
    if ((s = timer_begin(c.o.timing)) != WINGSPAN_OK) return s;
    c.dtype_f64 = dtype == WINGSPAN_F64 ? 1 : 0;
    if (dtype == WINGSPAN_F32)
        s = sharded_impl<float>(c, A, B, row_off_dev, row_nnz_dev, pool_col_dev, static_cast<float *>(pool_val_dev),
                                pool_capacity, pool_used);
    else
        s = sharded_impl<double>(c, A, B, row_off_dev, row_nnz_dev, pool_col_dev,
                                 static_cast<double *>(pool_val_dev), pool_capacity, pool_used);
    const wingspan_status t = finish_timing(2);
    return s != WINGSPAN_OK ? s : t;
}

wingspan_status wingspan_sharded_to_csr_workspace_size(int64_t nrows, size_t *bytes) {
    g_err.clear();
    if (!bytes) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bytes is NULL");
    if (nrows < 0 || nrows > INT32_MAX - 1) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "nrows out of range");
    const int64_t tiles = (nrows + 1 + kScanTile - 1) / kScanTile + 2;
    *bytes = align_up(sizeof(int64_t) * tiles);
    return WINGSPAN_OK;
}

wingspan_status wingspan_sharded_to_csr(int64_t nrows, int64_t nnz, const int64_t *row_off_dev, const int32_t *row_nnz_dev,
                                        const int32_t *pool_col_dev, const void *pool_val_dev, wingspan_dtype dtype,
                                        int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                        void *workspace_dev, size_t workspace_bytes, void *stream) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    size_t need = 0;
    wingspan_status s = wingspan_sharded_to_csr_workspace_size(nrows, &need);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if (nnz < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "nnz is negative");
    if (nnz > 0 && (!pool_col_dev || !pool_val_dev || !c_col_idx_dev || !c_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "a pool or C array is NULL");
    if (nrows > 0 && (!row_off_dev || !row_nnz_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "row_off_dev or row_nnz_dev is NULL");
    if (workspace_bytes < need)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
    if (!workspace_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(workspace_dev) % kAlign != 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kAlign);
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.partials = static_cast<int64_t *>(workspace_dev);
    if ((s = run_scan(c, CountIn{row_nnz_dev}, nrows, c_row_ptr_dev)) != WINGSPAN_OK) return s;
    if (nrows > 0 && nnz > 0) {
        const unsigned grid = static_cast<unsigned>((nnz + kGatherChunk - 1) / kGatherChunk);
        if (dtype == WINGSPAN_F32)
            gather_rows<float><<<grid, 256, 0, c.st>>>(nrows, row_off_dev, c_row_ptr_dev, pool_col_dev,
                                                       static_cast<const float *>(pool_val_dev), c_col_idx_dev,
                                                       static_cast<float *>(c_val_dev));
        else
            gather_rows<double><<<grid, 256, 0, c.st>>>(nrows, row_off_dev, c_row_ptr_dev, pool_col_dev,
                                                        static_cast<const double *>(pool_val_dev), c_col_idx_dev,
                                                        static_cast<double *>(c_val_dev));
        LAUNCH_CHECK("gather_rows");
    }
    return WINGSPAN_OK;
}

wingspan_status wingspan_elementwise_workspace_size(const wingspan_csr *A, const wingspan_csr *B, size_t *bytes) {
    g_err.clear();
    if (!bytes) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bytes is NULL");
    wingspan_status s = ew_check(WINGSPAN_OP_ADD, A, B);
    if (s != WINGSPAN_OK) return s;
    *bytes = ew_plan(A, B).total;
    return WINGSPAN_OK;
}

wingspan_status wingspan_elementwise_structure(wingspan_ew_op op, const wingspan_csr *A, const wingspan_csr *B,
                                               int64_t *c_row_ptr_dev, int64_t *c_nnz, void *workspace_dev,
                                               size_t workspace_bytes, void *stream) {
    g_err.clear();
    wingspan_status s = ew_check(op, A, B);
    if (s != WINGSPAN_OK) return s;
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if (!c_nnz) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_nnz is NULL");
    EwLayout L;
    if ((s = ew_workspace(A, B, workspace_dev, workspace_bytes, &L)) != WINGSPAN_OK) return s;
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.ws = static_cast<char *>(workspace_dev);
    const EwTiles T = ew_arrays(c, L);
    const int m = static_cast<int>(A->nrows);
    bool planned = false;
    ew_forget(workspace_dev, workspace_bytes);
    if (m > 0) {
        fill_i32<<<blocks_for(m, 256), 256, 0, c.st>>>(T.dups, m, 0);
        LAUNCH_CHECK("elementwise clear");
        // per-row common coordinates (none when a side is empty), and the tiles' places in C for the values
        if (A->nnz > 0 && B->nnz > 0) {
            if ((s = ew_count_tiles<true>(c, op, A, B, L, T)) != WINGSPAN_OK) return s;
            if ((s = ew_scan_tiles(c, L, T)) != WINGSPAN_OK) return s;
            planned = true;
        }
    }
    if ((s = run_scan(c, EwCountIn{A->row_ptr, B->row_ptr, T.dups, static_cast<int>(op)}, m, c_row_ptr_dev)) !=
        WINGSPAN_OK)
        return s;
    int64_t total = 0;
    HIP_TRY(hipMemcpyAsync(&total, c_row_ptr_dev + m, sizeof(int64_t), hipMemcpyDeviceToHost, c.st));
    HIP_TRY(hipStreamSynchronize(c.st));
    *c_nnz = total;
    if (planned) ew_remember(ew_key_of(op, A, B, workspace_dev, workspace_bytes));
    return WINGSPAN_OK;
}

wingspan_status wingspan_elementwise_values(wingspan_ew_op op, const wingspan_csr *A, const wingspan_csr *B,
                                            wingspan_dtype dtype, const int64_t *c_row_ptr_dev,
                                            int32_t *c_col_idx_dev, void *c_val_dev, void *workspace_dev,
                                            size_t workspace_bytes, void *stream) {
    g_err.clear();
    wingspan_status s = ew_check(op, A, B);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if ((A->nnz > 0 || B->nnz > 0) && (!c_col_idx_dev || !c_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_col_idx_dev or c_val_dev is NULL");
    EwLayout L;
    if ((s = ew_workspace(A, B, workspace_dev, workspace_bytes, &L)) != WINGSPAN_OK) return s;
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.ws = static_cast<char *>(workspace_dev);
    const EwPlanKey key = ew_key_of(op, A, B, workspace_dev, workspace_bytes);
    const bool planned = ew_known(key);
    if (!planned) ew_forget(workspace_dev, workspace_bytes);
    s = dtype == WINGSPAN_F32
            ? ew_values_impl<float>(c, op, A, B, L, c_col_idx_dev, static_cast<float *>(c_val_dev), planned)
            : ew_values_impl<double>(c, op, A, B, L, c_col_idx_dev, static_cast<double *>(c_val_dev), planned);
    if (s == WINGSPAN_OK && !planned && A->nrows > 0 && L.ntiles > 0 &&
        !(op == WINGSPAN_OP_HADAMARD && (A->nnz == 0 || B->nnz == 0)))
        ew_remember(key);
    return s;
}

wingspan_status wingspan_spmspv_workspace_size(const wingspan_csr *At, int64_t nnz_x, size_t *bytes) {
    g_err.clear();
    if (!bytes) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bytes is NULL");
    wingspan_status s = sv_check(At, nnz_x);
    if (s != WINGSPAN_OK) return s;
    *bytes = sv_plan(At, nnz_x).total;
    return WINGSPAN_OK;
}

wingspan_status wingspan_spmspv(const wingspan_csr *At, wingspan_dtype dtype, const int32_t *x_idx_dev,
                                const void *x_val_dev, int64_t nnz_x, int32_t *y_idx_dev, void *y_val_dev,
                                int64_t y_cap, int64_t *y_nnz, void *workspace_dev, size_t workspace_bytes,
                                void *stream) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    wingspan_status s = sv_check(At, nnz_x);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!y_nnz) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "y_nnz is NULL");
    if (nnz_x > 0 && (!x_idx_dev || !x_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "x has entries but x_idx_dev or x_val_dev is NULL");
    if (y_cap < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "y_cap is negative");
    if (y_cap > 0 && (!y_idx_dev || !y_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "y_cap > 0 but y_idx_dev or y_val_dev is NULL");
    const SvLayout L = sv_plan(At, nnz_x);
    if (workspace_bytes < L.total)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", workspace_bytes,
                    L.total);
    if (!workspace_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(workspace_dev) % kAlign != 0)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "workspace must be %zu-byte aligned", kAlign);
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.ws = static_cast<char *>(workspace_dev);
    c.partials = reinterpret_cast<int64_t *>(c.ws + L.off_partials);
    if (dtype == WINGSPAN_F32)
        return sv_impl<float>(c, At, L, x_idx_dev, static_cast<const float *>(x_val_dev), nnz_x, y_idx_dev,
                              static_cast<float *>(y_val_dev), y_cap, y_nnz);
    return sv_impl<double>(c, At, L, x_idx_dev, static_cast<const double *>(x_val_dev), nnz_x, y_idx_dev,
                           static_cast<double *>(y_val_dev), y_cap, y_nnz);
}

wingspan_status wingspan_outer_workspace_size(const wingspan_csr *At, const wingspan_csr *B, int64_t products,
                                              size_t *bytes) {
    g_err.clear();
    if (!bytes) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "bytes is NULL");
    wingspan_status s = op_check(At, B);
    if (s != WINGSPAN_OK) return s;
    if (products < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "products is negative");
    *bytes = op_plan(At, B, products).total;
    return WINGSPAN_OK;
}

wingspan_status wingspan_outer_products(const wingspan_csr *At, const wingspan_csr *B, int64_t *products,
                                        void *workspace_dev, size_t workspace_bytes, void *stream) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    wingspan_status s = op_check(At, B);
    if (s != WINGSPAN_OK) return s;
    if (!products) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "products is NULL");
    const OpLayout L = op_plan(At, B, 0);
    if ((s = op_workspace_ok(workspace_dev, workspace_bytes, L.off_part_key)) != WINGSPAN_OK) return s;
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.ws = static_cast<char *>(workspace_dev);
    return op_count(c, At, B, L, products);
}

wingspan_status wingspan_spgemm_outer(const wingspan_csr *At, const wingspan_csr *B, wingspan_dtype dtype,
                                      int64_t *c_row_ptr_dev, int32_t *c_col_idx_dev, void *c_val_dev,
                                      int64_t c_capacity, int64_t *c_nnz, void *workspace_dev, size_t workspace_bytes,
                                      void *stream) {
    g_err.clear();
    ew_forget(workspace_dev, workspace_bytes);   // a kept elementwise tiling is overwritten
    wingspan_status s = op_check(At, B);
    if (s != WINGSPAN_OK) return s;
    if (dtype != WINGSPAN_F32 && dtype != WINGSPAN_F64)
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "dtype must be WINGSPAN_F32 or WINGSPAN_F64");
    if (!c_nnz) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_nnz is NULL");
    if (!c_row_ptr_dev) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_row_ptr_dev is NULL");
    if (c_capacity < 0) return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_capacity is negative");
    if (c_capacity > 0 && (!c_col_idx_dev || !c_val_dev))
        return fail(WINGSPAN_ERR_INVALID_ARGUMENT, "c_capacity > 0 but c_col_idx_dev or c_val_dev is NULL");
    *c_nnz = 0;
    const OpLayout L0 = op_plan(At, B, 0);
    if ((s = op_workspace_ok(workspace_dev, workspace_bytes, L0.off_part_key)) != WINGSPAN_OK) return s;
    Ctx c{};
    c.st = static_cast<hipStream_t>(stream);
    c.ws = static_cast<char *>(workspace_dev);
    int64_t P = 0;
    if ((s = op_count(c, At, B, L0, &P)) != WINGSPAN_OK) return s;
    if (P > INT32_MAX)   // a row's count of partial entries is an int32
        return fail(WINGSPAN_ERR_UNSUPPORTED, "%lld products: the outer product takes at most %d",
                    (long long)P, INT32_MAX);
    const OpLayout L = op_plan(At, B, P);
    if (workspace_bytes < L.total)
        return fail(WINGSPAN_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed for %lld products",
                    workspace_bytes, L.total, (long long)P);
    if (dtype == WINGSPAN_F32)
        return op_impl<float>(c, At, B, L, P, c_row_ptr_dev, c_col_idx_dev, static_cast<float *>(c_val_dev),
                              c_capacity, c_nnz);
    return op_impl<double>(c, At, B, L, P, c_row_ptr_dev, c_col_idx_dev, static_cast<double *>(c_val_dev),
                           c_capacity, c_nnz);
}

}  // extern "C"
