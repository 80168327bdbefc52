// Host-only: how the N-sized passes of a launch group are split over
// workgroups.  Plain C++ (no HIP types), so it also builds in a host test.
#pragma once
#include <algorithm>
#include <cstdint>

namespace edkm {

// Split `count` matrices of n[i] weights over at most `budget` workgroups, in
// proportion to size by largest remainder (so the shares never add up to more
// than the budget), at least one workgroup per matrix and at most one per
// `min_chunk` weights.  Matrix i gets wg_count[i] workgroups starting at grid
// index wg_begin[i], each a slice of chunk[i] weights (a multiple of 8; the
// last slice may be short).  Returns the grid size, sum of wg_count.  Exceeds
// the budget only when count > budget.
inline uint32_t split_passes(const uint64_t* n, int count, int budget, uint64_t min_chunk,
                             uint64_t* chunk, uint32_t* wg_count, uint32_t* wg_begin) {
    constexpr int MAXC = 64;
    if (count < 1 || count > MAXC || budget < 1) return 0;
    double total = 0.0;
    for (int i = 0; i < count; ++i) total += (double)n[i];
    int64_t a[MAXC], cap[MAXC];
    double rem[MAXC];
    int64_t sum = 0;
    for (int i = 0; i < count; ++i) {
        cap[i] = (int64_t)std::min<uint64_t>((n[i] + min_chunk - 1) / min_chunk, (uint64_t)budget);
        if (cap[i] < 1) cap[i] = 1;
        const double q = (double)budget * (double)n[i] / total;
        a[i] = std::max<int64_t>(1, std::min<int64_t>((int64_t)q, cap[i]));
        rem[i] = q - (double)a[i];
        sum += a[i];
    }
    while (sum > budget) {          // only the one-per-matrix minimum can overshoot
        int j = -1;
        for (int i = 0; i < count; ++i)
            if (a[i] > 1 && (j < 0 || a[i] > a[j])) j = i;
        if (j < 0) break;
        --a[j];
        rem[j] += 1.0;
        --sum;
    }
    while (sum < budget) {          // hand out what is left by largest remainder
        int j = -1;
        for (int i = 0; i < count; ++i)
            if (a[i] < cap[i] && (j < 0 || rem[i] > rem[j])) j = i;
        if (j < 0) break;
        ++a[j];
        rem[j] -= 1.0;
        ++sum;
    }
    uint32_t wg = 0;
    for (int i = 0; i < count; ++i) {
        uint64_t c = (n[i] + (uint64_t)a[i] - 1) / (uint64_t)a[i];
        c = (c + 7) & ~7ull;
        chunk[i] = c;
        wg_count[i] = (uint32_t)((n[i] + c - 1) / c);
        wg_begin[i] = wg;
        wg += wg_count[i];
    }
    return wg;
}

}  // namespace edkm
