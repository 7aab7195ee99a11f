// Tile geometry of the radix sort, shared with the kernels that produce the
// keys: a producer whose workgroup b writes keys [b * kSortTile,
// (b + 1) * kSortTile) can count the first pass's digits of its tile as it
// goes (Pass0Hist), which saves the sort one read of the keys.
#pragma once

#include "expand.h"
#include "internal.h"

namespace gs {

// Build-time tunables: keys per thread of a sort tile (the emit's tile
// follows) and the widest digit of a pass.
#ifndef GS_SORT_ITEMS
#define GS_SORT_ITEMS 8
#endif
#ifndef GS_RADIX_BITS
#define GS_RADIX_BITS 10
#endif
constexpr int kSortItems = GS_SORT_ITEMS;
constexpr int kSortTile = kBlock * kSortItems;  // 2048
constexpr int kMaxDigitBits = GS_RADIX_BITS;
constexpr int kMaxDigits = 1 << kMaxDigitBits;
static_assert(kSortTile == kExpandTile, "emit tiles are sort tiles");
// Sorts of at least kBigSort pairs take tiles of kBigItems keys a thread
// (measured on a 22 M-pair index sort: 0.11 ms faster a sort; on 4 M pairs
// the longer tiles leave the chip under-filled).
constexpr int kBigItems = 2 * kSortItems;
constexpr int64_t kBigSort = (int64_t)1 << 23;

struct Pass0Hist {
    uint32_t *h;  // LDS, kMaxDigits words
    RadixPass0 p;
    __device__ __forceinline__ Pass0Hist(uint32_t *lds, const RadixPass0 &pass0) : h(lds), p(pass0) {
        if (p.table)
            for (uint32_t d = threadIdx.x; d <= p.mask; d += kBlock) h[d] = 0;
        __syncthreads();
    }
    __device__ __forceinline__ void add(uint32_t key) {
        if (p.table) atomicAdd(&h[key & p.mask], 1u);
    }
    // tile: the index of the tile this workgroup produced
    __device__ __forceinline__ void finish_tile(uint32_t tile) {
        __syncthreads();
        if (p.table)
            for (uint32_t d = threadIdx.x; d <= p.mask; d += kBlock) p.table[(size_t)d * p.nb + tile] = h[d];
    }
};

}  // namespace gs
