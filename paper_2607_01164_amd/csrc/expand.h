// Load-balanced expansion of segments: given exclusive offsets off[0..n]
// (segment g owns elements [off[g], off[g+1])), every workgroup takes a tile
// of consecutive elements and finds the owning segment of each element
// without a per-element search: segment starts inside the tile are marked
// in LDS and an inclusive max-scan carries them forward.
#pragma once

#include "internal.h"

namespace gs {

constexpr int kExpandItems = 8;
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

struct ExpandShared {
    uint32_t head[kExpandTile];
    int64_t seg_range[2];
    uint32_t wmax[kWavesPerBlock];
};

// Fills sh.head[s] with (owning segment - first segment of the tile) for the
// tile_cnt elements starting at tile_begin; returns the first segment.
// Must be called by the whole workgroup.
template <typename T>
__device__ __forceinline__ int64_t expand_tile(const T *__restrict__ off, int64_t nseg, uint64_t tile_begin,
                                               uint32_t tile_cnt, ExpandShared &sh) {
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    if (tid == 0) sh.seg_range[0] = segment_search(off, nseg, tile_begin);
    if (tid == 1) sh.seg_range[1] = segment_search(off, nseg, tile_begin + tile_cnt - 1);
    for (uint32_t s = tid; s < (uint32_t)kExpandTile; s += kBlock) sh.head[s] = 0;
    __syncthreads();
    const int64_t gfirst = sh.seg_range[0], glast = sh.seg_range[1];
    for (int64_t gg = gfirst + 1 + tid; gg <= glast; gg += kBlock) {
        const uint32_t pos = (uint32_t)((uint64_t)off[gg] - tile_begin);
        atomicMax(&sh.head[pos], (uint32_t)(gg - gfirst));
    }
    __syncthreads();
    uint32_t run = 0;
    const uint32_t b0 = tid * kExpandItems;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t h = sh.head[b0 + i];
        run = h > run ? h : run;
        sh.head[b0 + i] = run;
    }
    const uint32_t incl = wave_incl_max(run);
    uint32_t excl = __shfl_up(incl, 1, 64);
    if (lane == 0) excl = 0;
    if (lane == kWave - 1) sh.wmax[wave] = incl;
    __syncthreads();
    uint32_t wpre = 0;
    for (uint32_t w = 0; w < wave; ++w) wpre = sh.wmax[w] > wpre ? sh.wmax[w] : wpre;
    const uint32_t carry = excl > wpre ? excl : wpre;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t h = sh.head[b0 + i];
        sh.head[b0 + i] = h > carry ? h : carry;
    }
    __syncthreads();
    return gfirst;
}

}  // namespace gs
