// Searches shared by the flat (product- or entry-parallel) kernels: over
// prefix arrays, and merge-path splits of two sorted sequences.
#pragma once

#include "device_common.hpp"

namespace wsp {

// Last t in [0, n) with pref[t] <= q, for a non-decreasing pref with
// pref[0] <= q: a 64-ary search in which all 64 lanes of one wave take part
// (three rounds for a quarter million entries).
__device__ __forceinline__ int wave_find_entry(const int64_t *__restrict__ pref, int n, int64_t q) {
    int lo = 0, hi = n - 1;   // pref[lo] <= q holds throughout
    while (hi > lo) {
        const int step = (hi - lo + kWave) / kWave;
        const int idx = lo + lane_id() * step;
        const bool le = idx <= hi && pref[idx] <= q;
        const uint64_t m = ballot(le);
        lo = lo + (63 - __clzll(m)) * step;
        const int h = lo + step - 1;
        hi = h < hi ? h : hi;
    }
    return lo;
}

// The same search in an LDS copy: last index in [0, n) with s[idx] <= q.
__device__ __forceinline__ int lds_find_entry(const int64_t *s, int n, int64_t q) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s[mid] <= q) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Last r in [lo, hi] with f(r) <= q, for a non-decreasing f with f(lo) <= q:
// a 64-ary search in which all 64 lanes of one wave take part.
template <typename F>
__device__ __forceinline__ int wave_last_le(F f, int lo, int hi, int64_t q) {
    while (hi > lo) {
        const int64_t step = (static_cast<int64_t>(hi) - lo + kWave) / kWave;
        const int64_t idx = lo + lane_id() * step;
        const bool le = idx <= hi && f(static_cast<int>(idx)) <= q;
        const uint64_t m = ballot(le);   // lane 0 always qualifies
        lo = static_cast<int>(lo + (63 - __clzll(m)) * step);
        const int64_t h = lo + step - 1;
        hi = h < hi ? static_cast<int>(h) : hi;
    }
    return lo;
}

// Merge-path split of the stable merge of sorted a[0, na) and b[0, nb), a's
// entries first among equal keys: the number of a's entries among the first d
// outputs, i.e. the least i in [max(0, d - nb), min(d, na)] with
// i = min(d, na) or a[i] > b[d - i - 1]. One wave (all 64 lanes call it)
// evaluates 64 candidates per round; every lane returns the split.
__device__ inline int64_t wave_merge_split(const int32_t *a, int64_t na, const int32_t *b, int64_t nb, int64_t d) {
    int64_t lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
    while (lo < hi) {
        // lane l probes lo + (hi - lo) l / 64, all in [lo, hi): a[p] and b[d - p - 1] are in range
        const int64_t span = hi - lo;
        const int64_t p = lo + span * lane_id() / kWave;
        const uint64_t t = ballot(a[p] > b[d - p - 1]);
        if (t == 0ull) {
            lo += span * (kWave - 1) / kWave + 1;
        } else {
            const int l = __ffsll(static_cast<long long>(t)) - 1;
            hi = lo + span * l / kWave;
            lo = l == 0 ? lo : lo + span * (l - 1) / kWave + 1;
        }
    }
    return lo;
}

}  // namespace wsp
