// Device-wide primitives: exclusive scans, a stable LSD radix sort of
// (key, value) pairs with wave-level multi-split ranking in LDS, per-key
// offsets of a sorted key array, and fills.
#include "internal.h"
#include "radix.h"

namespace gs {

namespace {

constexpr int kScanItems = 16;
constexpr int kScanTile = kBlock * kScanItems;  // 4096

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_reduce(const T *__restrict__ in, int64_t n, T *__restrict__ sums) {
    __shared__ T lds[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    T s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        int64_t idx = base + i;
        if (idx < n) s += in[idx];
    }
    T tot;
    (void)block_excl_scan(s, lds, &tot);
    if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_tile(const T *in, T *out, int64_t n, const T *__restrict__ prefix,
                                                      T *__restrict__ total) {
    __shared__ T lds[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    T v[kScanItems];
    T s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        int64_t idx = base + i;
        v[i] = idx < n ? in[idx] : T(0);
        s += v[i];
    }
    T tot;
    T run = block_excl_scan(s, lds, &tot);
    if (prefix) run += prefix[blockIdx.x];
    // the last workgroup's last thread ends with the grand total
    if (total && blockIdx.x == gridDim.x - 1 && threadIdx.x == kBlock - 1) *total = run + s;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        int64_t idx = base + i;
        if (idx < n) out[idx] = run;
        run += v[i];
    }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// total (optional) receives the sum of all n elements
template <typename T>
hipError_t scan_rec(const T *in, T *out, int64_t n, T *work, hipStream_t s, T *total = nullptr) {
    if (n <= 0) return hipSuccess;
    if (n <= kScanTile) {
        hipLaunchKernelGGL(k_scan_tile<T>, dim3(1), dim3(kBlock), 0, s, in, out, n, (const T *)nullptr, total);
        return hipGetLastError();
    }
    const int64_t nb = ceil_div(n, kScanTile);
    T *sums = work;
    hipLaunchKernelGGL(k_scan_reduce<T>, dim3((uint32_t)nb), dim3(kBlock), 0, s, in, n, sums);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = scan_rec<T>(sums, sums, nb, work + nb, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_tile<T>, dim3((uint32_t)nb), dim3(kBlock), 0, s, in, out, n, (const T *)sums, total);
    return hipGetLastError();
}

int64_t scan_levels_elems(int64_t n) {
    int64_t tot = 0;
    while (n > kScanTile) {
        n = ceil_div(n, kScanTile);
        tot += n;
    }
    return tot;
}

// ---------------------------------------------------------------------------
// Radix sort (stable LSD, reduce-then-scan). Per pass: tile histograms of
// the digit (the first pass's can come from the kernel that produced the
// keys), an exclusive scan of every digit's row of tile counts that also
// yields the digit totals, and a scatter that scans the totals, ranks its
// tile in LDS and writes it out digit by digit.

int passes_for(int bits) { return bits <= 0 ? 0 : (bits + kMaxDigitBits - 1) / kMaxDigitBits; }
int digit_bits_for(int bits) {
    int p = passes_for(bits);
    return p == 0 ? 0 : (bits + p - 1) / p;
}

template <int ITEMS>
__global__ __launch_bounds__(kBlock) void k_radix_upsweep(const uint32_t *__restrict__ keys, int64_t n, int shift,
                                                          uint32_t mask, uint32_t ndig, uint32_t *__restrict__ table,
                                                          uint32_t nb) {
    __shared__ uint32_t h[kMaxDigits];
    for (uint32_t d = threadIdx.x; d < ndig; d += kBlock) h[d] = 0;
    __syncthreads();
    const uint32_t tile = xcd_block(blockIdx.x, gridDim.x);
    const int64_t base = (int64_t)tile * (kBlock * ITEMS);
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + (int64_t)i * kBlock + threadIdx.x;
        if (idx < n) atomicAdd(&h[(keys[idx] >> shift) & mask], 1u);
    }
    __syncthreads();
    for (uint32_t d = threadIdx.x; d < ndig; d += kBlock) table[(size_t)d * nb + tile] = h[d];
}

// One workgroup per digit: exclusive scan of the digit's tile counts in
// place, and the digit's total.
__global__ __launch_bounds__(kBlock) void k_digit_scan(uint32_t *__restrict__ table, uint32_t nb,
                                                       uint32_t *__restrict__ digit_tot) {
    __shared__ uint32_t lds[kWavesPerBlock];
    uint32_t *row = table + (size_t)blockIdx.x * nb;
    uint32_t carry = 0;
    for (uint32_t c0 = 0; c0 < nb; c0 += kBlock * 4) {
        uint32_t v[4];
        uint32_t s = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t idx = c0 + threadIdx.x * 4 + i;
            v[i] = idx < nb ? row[idx] : 0u;
            s += v[i];
        }
        uint32_t tot;
        uint32_t run = block_excl_scan(s, lds, &tot) + carry;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t idx = c0 + threadIdx.x * 4 + i;
            if (idx < nb) row[idx] = run;
            run += v[i];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) digit_tot[blockIdx.x] = carry;
}

// Stable scatter of one tile of 64 ITEMS keys. Each wave ranks its ITEMS
// rows of 64 keys in order: lanes holding the same digit are found with one
// ballot per digit bit, and a per-wave running count per digit in LDS gives
// each key its rank among earlier keys of the wave. Waves are then combined
// per digit, the tile is reordered by digit in LDS and written out in runs.
// The tile's place in each digit's row of the table is column tile <<
// col_shift (a first pass counted by the keys' producer in tiles half as
// long has col_shift 1). LDS: (2 ndig + 2 TILE) words, dynamic.
template <int ITEMS>
__global__ __launch_bounds__(kBlock) void k_radix_downsweep(const uint32_t *__restrict__ kin,
                                                            const uint32_t *__restrict__ vin,
                                                            uint32_t *__restrict__ kout, uint32_t *__restrict__ vout,
                                                            int64_t n, int shift, int dbits,
                                                            const uint32_t *__restrict__ table,
                                                            const uint32_t *__restrict__ digit_tot, uint32_t nb,
                                                            int col_shift) {
    constexpr int TILE = kBlock * ITEMS;
    extern __shared__ uint32_t lds[];
    __shared__ uint32_t scan_lds[kWavesPerBlock];
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const uint32_t ndig = 1u << dbits, mask = ndig - 1;
    // consecutive tiles on one XCD: their runs of each digit are adjacent in
    // the output and merge in that XCD's L2
    const uint32_t tile = xcd_block(blockIdx.x, gridDim.x);
    uint32_t *dstart = lds;                      // [ndig]
    uint32_t *dglob = dstart + ndig;             // [ndig]
    uint32_t *sk = dglob + ndig;                 // [TILE]
    uint32_t *sv = sk + TILE;                    // [TILE]
    // the per-wave digit counts share the tile buffers' space: they are all
    // read before the tile is written there (kWavesPerBlock ndig <= 2 TILE)
    uint32_t *wcnt = sk;                         // [kWavesPerBlock][ndig]
    const int64_t base = (int64_t)tile * TILE + (int64_t)wave * (kWave * ITEMS);
    uint32_t k[ITEMS], v[ITEMS], r[ITEMS];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + (int64_t)i * kWave + lane;
        const bool ok = idx < n;
        k[i] = ok ? kin[idx] : 0u;
        v[i] = ok ? vin[idx] : 0u;
    }
    // output start of every digit in this tile: the exclusive scan of the
    // digit totals plus the tile's place in its digit's row (all loads are
    // issued before the first wait)
    constexpr int J = kMaxDigits > kBlock ? kMaxDigits / kBlock : 1;
    uint32_t loc[J], tpre[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const uint32_t d = tid * J + j;
        loc[j] = d < ndig ? digit_tot[d] : 0u;
        tpre[j] = d < ndig ? table[(size_t)d * nb + ((size_t)tile << col_shift)] : 0u;
    }
    for (uint32_t d = tid; d < ndig; d += kBlock) {
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) wcnt[w * ndig + d] = 0;
    }
    {
        uint32_t s = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) s += loc[j];
        uint32_t tot;
        uint32_t run = block_excl_scan(s, scan_lds, &tot);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const uint32_t d = tid * J + j;
            if (d < ndig) dglob[d] = run + tpre[j];
            run += loc[j];
        }
    }
    __syncthreads();

    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t *mycnt = wcnt + wave * ndig;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + (int64_t)i * kWave + lane;
        const bool ok = idx < n;
        const uint32_t d = (k[i] >> shift) & mask;
        uint64_t m = __ballot(ok);
        for (int b = 0; b < dbits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bm = __ballot(bit);
            m &= bit ? bm : ~bm;
        }
        const uint32_t before = (uint32_t)__popcll(m & lt_mask);
        const uint32_t cnt = (uint32_t)__popcll(m);
        uint32_t basecnt = 0;
        if (ok) basecnt = mycnt[d];
        // every lane of the wave has read the counter before its leader writes
        __builtin_amdgcn_wave_barrier();
        if (ok && before == 0) mycnt[d] = basecnt + cnt;
        __builtin_amdgcn_wave_barrier();
        r[i] = basecnt + before;
    }
    __syncthreads();
    // per digit: exclusive scan over the waves (in place) and the tile total
    for (uint32_t d = tid; d < ndig; d += kBlock) {
        uint32_t s = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) {
            const uint32_t t = wcnt[w * ndig + d];
            wcnt[w * ndig + d] = s;
            s += t;
        }
        dstart[d] = s;
    }
    __syncthreads();
    {
        uint32_t loc[J];
        uint32_t s = 0;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const uint32_t d = tid * J + j;
            loc[j] = d < ndig ? dstart[d] : 0u;
            s += loc[j];
        }
        uint32_t tot;
        uint32_t run = block_excl_scan(s, scan_lds, &tot);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const uint32_t d = tid * J + j;
            if (d < ndig) dstart[d] = run;
            run += loc[j];
        }
    }
    __syncthreads();
    uint32_t slot[ITEMS];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + (int64_t)i * kWave + lane;
        const uint32_t d = (k[i] >> shift) & mask;
        slot[i] = idx < n ? dstart[d] + mycnt[d] + r[i] : 0u;
    }
    // every counter is read before the tile overwrites their space
    __syncthreads();
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + (int64_t)i * kWave + lane;
        if (idx < n) {
            sk[slot[i]] = k[i];
            sv[slot[i]] = v[i];
        }
    }
    __syncthreads();
    const int64_t tile_n = n - (int64_t)tile * TILE;
    const uint32_t cnt = tile_n < TILE ? (uint32_t)tile_n : (uint32_t)TILE;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
        const uint32_t slot = (uint32_t)i * kBlock + tid;
        if (slot < cnt) {
            const uint32_t key = sk[slot];
            const uint32_t d = (key >> shift) & mask;
            const uint32_t pos = dglob[d] + (slot - dstart[d]);
            if ((int64_t)pos < n) {
                kout[pos] = key;
                vout[pos] = sv[slot];
            }
        }
    }
}

// Exclusive scan of per-segment counts into offsets, in place, for counts
// whose sums over groups of kPairSumGroup elements were scanned already
// (group_prefix, with the grand total after the last group): workgroup b
// takes kPairTile elements and starts at group_prefix[b kPairTile / 64].
// Every non-empty segment i also records itself as the first segment of the
// tiles of tile_size elements that start inside it.
constexpr int kPairSumGroup = 64;
constexpr int kPairItems = 4;
constexpr int kPairTile = kBlock * kPairItems;  // 1024
static_assert(kPairTile % kPairSumGroup == 0, "offset tiles are whole groups");
__global__ __launch_bounds__(kBlock) void k_pair_offsets(uint64_t *__restrict__ off, int64_t n,
                                                         const uint64_t *__restrict__ group_prefix,
                                                         uint32_t *__restrict__ tile_first, int64_t ntiles,
                                                         uint32_t tile_size) {
    __shared__ uint64_t lds[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kPairTile + (int64_t)threadIdx.x * kPairItems;
    uint64_t v[kPairItems];
    uint64_t s = 0;
#pragma unroll
    for (int i = 0; i < kPairItems; ++i) {
        const int64_t idx = base + i;
        v[i] = idx < n ? off[idx] : 0ull;
        s += v[i];
    }
    uint64_t tot;
    uint64_t run = block_excl_scan(s, lds, &tot) + group_prefix[(size_t)blockIdx.x * (kPairTile / kPairSumGroup)];
#pragma unroll
    for (int i = 0; i < kPairItems; ++i) {
        const int64_t idx = base + i;
        if (idx < n) {
            off[idx] = run;
            if (v[i] > 0) {
                const uint64_t t0 = (run + tile_size - 1) / tile_size, t1 = (run + v[i] - 1) / tile_size;
                for (uint64_t t = t0; t <= t1 && t < (uint64_t)ntiles; ++t) tile_first[t] = (uint32_t)idx;
            }
        }
        run += v[i];
    }
}

// offsets[k] = number of keys < k, for k = 0 .. nkeys. Wave w covers keys
// k0 = 64 w .. k0 + 63. It first bounds all of them at once: lanes 0..31
// search for the first sorted key >= k0 and lanes 32..63 for the first >= k0
// + 64, each half probing 32 evenly spaced keys of its interval a step
// (about log32(n) dependent loads, where a binary search takes log2(n)).
// Lane l then finds its own key k0 + l by binary search between the two,
// inside one short stretch of the array that the wave's lanes share. The
// cost of a wave does not depend on how long runs of empty keys are.
__global__ __launch_bounds__(kBlock) void k_key_offsets(const uint32_t *__restrict__ keys, int64_t n,
                                                        uint32_t *__restrict__ off, int64_t nkeys) {
    const uint32_t lane = threadIdx.x % kWave;
    const int64_t k0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) - lane;
    if (k0 > nkeys) return;  // whole waves leave together
    const bool upper = lane >= 32;
    const uint32_t l = lane & 31u;
    const int64_t t = upper ? k0 + 64 : k0;
    // the first index whose key is >= t lies in [lo, hi]
    uint64_t lo = 0, hi = (uint64_t)n;
    while (__ballot(hi > lo) != 0) {
        const uint64_t len = hi - lo;
        const uint64_t step = (len + 31) / 32;
        const uint64_t p = lo + (uint64_t)l * step;
        const bool less = p < hi && (int64_t)keys[p] < t;
        const uint64_t m = __ballot(less);
        const uint32_t cnt = (uint32_t)__popcll(upper ? (m >> 32) : (m & 0xffffffffull));
        if (hi > lo) {
            if (cnt == 0) {
                hi = lo;
            } else {
                const uint64_t last = lo + (uint64_t)(cnt - 1) * step;  // its key is < t
                const uint64_t next = last + step;                       // its key is >= t, if probed
                lo = last + 1;
                if (next < hi) hi = next;
            }
        }
    }
    const uint64_t a = (uint64_t)__shfl((int)(uint32_t)lo, 0, kWave) |
                       ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(lo >> 32), 0, kWave) << 32);
    const uint64_t b = (uint64_t)(uint32_t)__shfl((int)(uint32_t)lo, 32, kWave) |
                       ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(lo >> 32), 32, kWave) << 32);
    const int64_t k = k0 + lane;
    uint64_t first = a, len = b - a;
    while (len > 0) {
        const uint64_t half = len >> 1;
        if ((int64_t)keys[first + half] < k) {
            first += half + 1;
            len -= half + 1;
        } else {
            len = half;
        }
    }
    if (k <= nkeys) off[k] = (uint32_t)first;
}

__global__ void k_fill_u32(uint32_t *p, uint32_t v, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_fill_f32(float *p, float v, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

}  // namespace

size_t scan_work_bytes(int64_t n, int elem_bytes) {
    return (size_t)(scan_levels_elems(n) + 1) * (size_t)elem_bytes;
}

hipError_t exclusive_scan_u32(const uint32_t *in, uint32_t *out, int64_t n, void *work, hipStream_t s) {
    prof_begin("scan_u32", s);
    hipError_t e = scan_rec<uint32_t>(in, out, n, (uint32_t *)work, s);
    prof_end("scan_u32", s);
    return e;
}

hipError_t pair_offsets(uint64_t *count, int64_t n, const uint64_t *group_prefix, uint32_t *tile_first,
                        int64_t ntiles, uint32_t tile_size, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    prof_begin("pair_offsets", s);
    hipLaunchKernelGGL(k_pair_offsets, dim3((uint32_t)ceil_div(n, kPairTile)), dim3(kBlock), 0, s, count, n,
                       group_prefix, tile_first, ntiles, tile_size);
    prof_end("pair_offsets", s);
    return hipGetLastError();
}

hipError_t exclusive_scan_u64_total(const uint64_t *in, uint64_t *out, int64_t n, uint64_t *total, void *work,
                                    hipStream_t s) {
    prof_begin("scan_u64", s);
    hipError_t e = scan_rec<uint64_t>(in, out, n, (uint64_t *)work, s, total);
    prof_end("scan_u64", s);
    return e;
}

hipError_t exclusive_scan_u64(const uint64_t *in, uint64_t *out, int64_t n, void *work, hipStream_t s) {
    prof_begin("scan_u64", s);
    hipError_t e = scan_rec<uint64_t>(in, out, n, (uint64_t *)work, s);
    prof_end("scan_u64", s);
    return e;
}

int radix_passes(int bits) { return passes_for(bits); }

RadixLayout radix_layout(void *work, int64_t n, int bits) {
    RadixLayout L;
    L.passes = passes_for(bits);
    L.dbits = digit_bits_for(bits);
    L.nb = (uint32_t)ceil_div(n > 0 ? n : 1, kSortTile);
    const uint32_t ndig = L.dbits > 0 ? (1u << L.dbits) : 1u;
    char *b = (char *)work;
    L.table = (uint32_t *)b;
    const size_t tbytes = ((size_t)ndig * L.nb * 4 + 255) & ~(size_t)255;
    L.digit_tot = b ? (uint32_t *)(b + tbytes) : nullptr;
    L.bytes = tbytes + (((size_t)ndig * 4 + 255) & ~(size_t)255);
    return L;
}

size_t radix_work_bytes(int64_t n, int bits) { return radix_layout(nullptr, n, bits).bytes; }

RadixPass0 radix_pass0(void *work, int64_t n, int bits) {
    const RadixLayout L = radix_layout(work, n, bits);
    RadixPass0 p;
    p.table = L.passes > 0 ? L.table : nullptr;
    p.nb = L.nb;
    p.mask = L.dbits > 0 ? (1u << L.dbits) - 1u : 0u;
    return p;
}

// Sorts n pairs that start in (k0, v0); passes alternate between (k0, v0)
// and (k1, v1). The result is in (k0, v0) after an even number of passes
// and in (k1, v1) after an odd number (radix_passes(bits)). When pass0_ready
// the producer of the keys has already written the first pass's tile
// histograms (radix_pass0, tiles of kSortTile keys). From kBigSort pairs
// the passes take tiles of kBigItems keys a thread: half as many tiles,
// each writing runs twice as long, and half the table to scan.
hipError_t radix_sort_pairs(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n, int bits, void *work,
                            hipStream_t s, bool pass0_ready) {
    const RadixLayout L = radix_layout(work, n, bits);
    if (L.passes == 0 || n <= 0) return hipSuccess;
    if (n == 1) {
        // already sorted; move it where an odd number of passes would leave it
        if (L.passes & 1) {
            hipError_t e = hipMemcpyAsync(k1, k0, 4, hipMemcpyDeviceToDevice, s);
            if (e == hipSuccess) e = hipMemcpyAsync(v1, v0, 4, hipMemcpyDeviceToDevice, s);
            return e;
        }
        return hipSuccess;
    }
    const uint32_t ndig = 1u << L.dbits;
    static_assert(kWavesPerBlock * kMaxDigits <= 2 * kSortTile, "the wave counts fit the tile buffers");
    static_assert(kBigItems % kSortItems == 0 && kBigItems / kSortItems == 2, "a big tile is two producer tiles");
    const bool big = n >= kBigSort;
    const int items = big ? kBigItems : kSortItems;
    const uint32_t ntiles = (uint32_t)ceil_div(n, (int64_t)kBlock * items);
    const size_t lds = ((size_t)2 * ndig + 2 * (size_t)kBlock * items) * 4;
    uint32_t *ki = k0, *vi = v0, *ko = k1, *vo = v1;
    for (int p = 0; p < L.passes; ++p) {
        const int shift = p * L.dbits;
        hipError_t e;
        // the table's columns this pass: the producer's tiles (a first pass
        // it counted) or the sort's own
        uint32_t ncols = ntiles;
        int col_shift = 0;
        if (p == 0 && pass0_ready) {
            ncols = L.nb;
            col_shift = big ? 1 : 0;
        } else {
            prof_begin("radix_upsweep", s);
            if (big)
                hipLaunchKernelGGL(k_radix_upsweep<kBigItems>, dim3(ntiles), dim3(kBlock), 0, s, ki, n, shift,
                                   ndig - 1, ndig, L.table, ncols);
            else
                hipLaunchKernelGGL(k_radix_upsweep<kSortItems>, dim3(ntiles), dim3(kBlock), 0, s, ki, n, shift,
                                   ndig - 1, ndig, L.table, ncols);
            prof_end("radix_upsweep", s);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        prof_begin("radix_scan", s);
        hipLaunchKernelGGL(k_digit_scan, dim3(ndig), dim3(kBlock), 0, s, L.table, ncols, L.digit_tot);
        prof_end("radix_scan", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        prof_begin("radix_downsweep", s);
        if (big)
            hipLaunchKernelGGL(k_radix_downsweep<kBigItems>, dim3(ntiles), dim3(kBlock), lds, s, ki, vi, ko, vo, n,
                               shift, L.dbits, L.table, L.digit_tot, ncols, col_shift);
        else
            hipLaunchKernelGGL(k_radix_downsweep<kSortItems>, dim3(ntiles), dim3(kBlock), lds, s, ki, vi, ko, vo, n,
                               shift, L.dbits, L.table, L.digit_tot, ncols, col_shift);
        prof_end("radix_downsweep", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        uint32_t *tk = ki, *tv = vi;
        ki = ko;
        vi = vo;
        ko = tk;
        vo = tv;
    }
    return hipSuccess;
}

hipError_t key_offsets(const uint32_t *sorted_keys, int64_t n, uint32_t *offsets, int64_t nkeys, hipStream_t s) {
    const int64_t threads = nkeys + 1;
    prof_begin("key_offsets", s);
    hipLaunchKernelGGL(k_key_offsets, dim3((uint32_t)ceil_div(threads, kBlock)), dim3(kBlock), 0, s, sorted_keys, n,
                       offsets, nkeys);
    prof_end("key_offsets", s);
    return hipGetLastError();
}

hipError_t fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_u32, dim3((uint32_t)ceil_div(n, kBlock)), dim3(kBlock), 0, s, p, v, n);
    return hipGetLastError();
}

hipError_t fill_f32(float *p, float v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_f32, dim3((uint32_t)ceil_div(n, kBlock)), dim3(kBlock), 0, s, p, v, n);
    return hipGetLastError();
}

}  // namespace gs
