// Tiles of consecutive elements of a segmented list (the pair emission and
// the sort share the tile size) and the owning-segment search: given
// exclusive offsets off[0..n] (segment g owns elements [off[g], off[g+1])),
// the segment of an element.
#pragma once

#include "internal.h"

namespace gs {

#ifndef GS_SORT_ITEMS
#define GS_SORT_ITEMS 8
#endif
constexpr int kExpandItems = GS_SORT_ITEMS;
constexpr int kExpandTile = kBlock * kExpandItems;  // 2048 elements per workgroup

// largest g in [0, n) with off[g] <= x (requires off[0] = 0 <= x)
template <typename T>
__device__ __forceinline__ int64_t segment_search(const T *__restrict__ off, int64_t n, uint64_t x) {
    int64_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if ((uint64_t)off[mid] <= x) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

}  // namespace gs
