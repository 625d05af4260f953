// Searches over prefix arrays shared by the flat (product- or entry-parallel)
// kernels.
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

}  // namespace wsp
