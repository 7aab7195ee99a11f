// Forward sampling (paper Eq. 2 with the cutoff test of Sec. 4.1.1 and the
// definedness rule of Sec. 4.1.3).
//
// Grid queries (Sec. 4.1.3, Fig. 4 C): one wavefront per (cell, 64 voxels of
// the cell); every lane is a voxel and all lanes walk the cell's Gaussian
// list together. The 48-byte Gaussian records are staged in the wave's LDS
// planes 64 at a time (the paper's shared-memory batches) and read there
// with one address for all lanes.
//
// Voxel-list and point queries (Sec. 5.1.2): the queries are first ordered
// by cell and, inside a cell, by quarter of the cell along x (query_keys +
// radix sort, kept in the plan) and the work is split by cell: dense cells run like grid cells, cells of fewer queries spread
// queries and candidates over the lanes (see k_sample_cells).
#include "expand.h"
#include "internal.h"
#include "radix.h"

#pragma clang fp contract(off)

namespace gs {

namespace {


// The samplers run one wave per workgroup. Their waves are independent
// (each has its own LDS buffer) and the cost of a work item varies by
// orders of magnitude with the cell's list and queries: a workgroup keeps
// its LDS until its slowest wave ends, so one-wave workgroups hand a
// finished wave's slot and LDS straight to new work. Work items are taken
// in launch order, which the dispatcher deals round-robin over the XCDs:
// with a fixed block-to-XCD remap, each XCD would own one contiguous
// stretch of cells, and clustered data would leave most XCDs idle while
// one works through the dense part.
constexpr int kSampWaves = 1;
constexpr int kSampBlock = kSampWaves * kWave;
constexpr int kSampPerSimd = 7;  // waves per SIMD the point sampler is compiled for

// Q' = Q log2(e) / 2 of a record at a point (record_q), G = 2^-Q'.
__device__ __forceinline__ float cutoff_q(const Record &r, float px, float py, float pz) {
    return record_q(r, px, py, pz);
}

__device__ __forceinline__ void accumulate(const Record &r, float px, float py, float pz, float T, float &I,
                                           float &V) {
    const float Q = cutoff_q(r, px, py, pz);
    if (Q <= T) {
        const float G = exp2_hw(-Q);
        I = fmaf_(r.f0.w, G, I);
        V = fmaf_(r.f1.w, G, V);
    }
}

// Records staged for the queries of one cell are rewritten relative to a
// point o of the cell (its centre): the first quarter of candidate s holds
// (-c, w) with c = U (mu - o), so that a query at a = p - o has u = U a - c,
// six FMAs where U (p - mu) takes three subtractions and six operations.
// Both offsets are at most a cell and a cutoff radius long, so u is formed
// from terms of its own size plus the cell's extent in units of the
// Gaussian's scale, and the rounding of Q' grows with that extent: on the
// five workloads' Gaussians near their cutoffs it stays within 0.15 of the
// float32 band of the cutoff the oracle allows (0.07 for U (p - mu)), but
// with cells a few hundred times a Gaussian's largest scale it leaves the
// band. The preprocess marks the cells of such Gaussians' boxes (cell
// diagonal above kOffsetCells times the largest scale), and the dense walk
// evaluates a marked cell as U (p - mu).
// Lane s rewrites candidate s of the wave's planes. The dense cells' walk
// takes it: with two queries a lane it is bound by VALU issue (10^8
// clustered points: the forward 6.6 % faster), and the items of one query a
// lane take it too so that both give the same bits. The grid cells' walk
// and the query rows are bound by their LDS reads; the rewrite made them
// 1-3 % slower, and they keep U (p - mu).
__device__ __forceinline__ void offset_planes(float4 *buf, uint32_t lane, float ox, float oy, float oz) {
    const float4 f0 = buf[lane], f1 = buf[kWave + lane], f2 = buf[2 * kWave + lane];
    const float bx = f0.x - ox, by = f0.y - oy, bz = f0.z - oz;
    const float c0 = fmaf_(f1.x, bx, fmaf_(f1.y, by, f1.z * bz));
    const float c1 = fmaf_(f2.x, by, f2.y * bz);
    const float c2 = f2.z * bz;
    buf[lane] = make_float4(-c0, -c1, -c2, f0.w);
}

// Q' of a rewritten record (f0 = (-c, w)) at the offset a = p - o.
__device__ __forceinline__ float offset_q(const Record &r, float ax, float ay, float az) {
    const float u0 = fmaf_(r.f1.x, ax, fmaf_(r.f1.y, ay, fmaf_(r.f1.z, az, r.f0.x)));
    const float u1 = fmaf_(r.f2.x, ay, fmaf_(r.f2.y, az, r.f0.y));
    const float u2 = fmaf_(r.f2.z, az, r.f0.z);
    return fmaf_(u0, u0, fmaf_(u1, u1, u2 * u2));
}

// The sums without a branch: G is selected (0 past the cutoff) and always
// added, so that a lane's queries cost one select each (adding w 0 and
// (w v) 0 leaves I and V as they are: both start at +0 and w, v are finite).
__device__ __forceinline__ void accumulate_sel(const Record &r, float px, float py, float pz, float T, float &I,
                                               float &V) {
    const float Q = cutoff_q(r, px, py, pz);
    const float G = Q <= T ? exp2_hw(-Q) : 0.0f;
    I = fmaf_(r.f0.w, G, I);
    V = fmaf_(r.f1.w, G, V);
}

__device__ __forceinline__ void accumulate_off_sel(const Record &r, float ax, float ay, float az, float T, float &I,
                                                   float &V) {
    const float Q = offset_q(r, ax, ay, az);
    const float G = Q <= T ? exp2_hw(-Q) : 0.0f;
    I = fmaf_(r.f0.w, G, I);
    V = fmaf_(r.f1.w, G, V);
}

// Four consecutive work items per XCD (xcd_group): the items of one cell
// share that XCD's L2 (C5's forward 1.6 % faster, C4's unchanged).
constexpr uint32_t kXcdItems = 4;

// The centre of cell c (float32; any point of the cell would do), for a
// wave-uniform c: kept in scalar registers.
__device__ __forceinline__ void cell_centre(const GridParams &g, uint32_t c, float &ox, float &oy, float &oz) {
    const uint32_t nx = (uint32_t)g.cells[0], ny = (uint32_t)g.cells[1];
    const uint32_t cx = c % nx, cy = (c / nx) % ny, cz = c / (nx * ny);
    ox = readfirst_f(g.lo[0] + ((float)cx + 0.5f) / g.invc[0]);
    oy = readfirst_f(g.lo[1] + ((float)cy + 0.5f) / g.invc[1]);
    oz = readfirst_f(g.lo[2] + ((float)cz + 0.5f) / g.invc[2]);
}

// Walk a wave-uniform candidate list [ja, jb) for one query per lane. The
// list is staged in the wave's LDS planes (buf: 3 planes of kWave float4) 64
// records at a time: lane l copies candidate c0 + l's record from memory
// straight into LDS (lanes past the list copy its last record), the ids of
// the next 64 are fetched meanwhile, and every lane then reads each record
// with the same address (a broadcast). One wait for memory per 64
// candidates, instead of a dependent id and record load per candidate.
__device__ __forceinline__ void walk_staged(const Record *__restrict__ rec, const uint32_t *__restrict__ gids,
                                            uint32_t ja, uint32_t jb, uint32_t lane, float4 *buf, float px,
                                            float py, float pz, float T, float &I, float &V) {
    uint32_t gnext = 0;
    if (ja < jb) gnext = gids[ja + lane < jb ? ja + lane : jb - 1];
    for (uint32_t c0 = ja; c0 < jb; c0 += kWave) {
        const float4 *src = (const float4 *)(rec + gnext);
#pragma unroll
        for (int qq = 0; qq < kRecordQuads; ++qq)
            __builtin_amdgcn_global_load_lds((const void *)(src + qq),
                                             (__attribute__((address_space(3))) void *)(buf + qq * kWave), 16, 0, 0);
        if (c0 + kWave < jb) gnext = gids[c0 + kWave + lane < jb ? c0 + kWave + lane : jb - 1];
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_wave_barrier();
        const uint32_t cnt = jb - c0 < (uint32_t)kWave ? jb - c0 : (uint32_t)kWave;
        uint32_t s = 0;
        for (; s + 2 <= cnt; s += 2) {
            Record a, b;
            a.f0 = buf[s];
            a.f1 = buf[kWave + s];
            a.f2 = buf[2 * kWave + s];
            b.f0 = buf[s + 1];
            b.f1 = buf[kWave + s + 1];
            b.f2 = buf[2 * kWave + s + 1];
            accumulate(a, px, py, pz, T, I, V);
            accumulate(b, px, py, pz, T, I, V);
        }
        if (s < cnt) {
            Record a;
            a.f0 = buf[s];
            a.f1 = buf[kWave + s];
            a.f2 = buf[2 * kWave + s];
            accumulate(a, px, py, pz, T, I, V);
        }
        // every lane has read the planes before the next chunk overwrites them
        __builtin_amdgcn_wave_barrier();
    }
}

// R queries per lane against a wave-uniform list [ja, jb), staged in the
// wave's LDS planes 64 records at a time as in walk_staged: each record
// read there serves the lane's R queries.
template <uint32_t R>
__device__ __forceinline__ void walk_staged_r(const Record *__restrict__ rec, bool off,
                                              const uint32_t *__restrict__ gids, uint32_t ja, uint32_t jb,
                                              uint32_t lane, float4 *buf,
                                              const float (&px)[R], const float (&py)[R], const float (&pz)[R],
                                              float ox, float oy, float oz, float T, float (&I)[R],
                                              float (&V)[R]) {
    float ax[R], ay[R], az[R];
#pragma unroll
    for (uint32_t t = 0; t < R; ++t) {
        ax[t] = px[t] - ox;
        ay[t] = py[t] - oy;
        az[t] = pz[t] - oz;
    }
    uint32_t gnext = 0;
    if (ja < jb) gnext = gids[ja + lane < jb ? ja + lane : jb - 1];
    for (uint32_t c0 = ja; c0 < jb; c0 += kWave) {
        const float4 *src = (const float4 *)(rec + gnext);
#pragma unroll
        for (int qq = 0; qq < kRecordQuads; ++qq)
            __builtin_amdgcn_global_load_lds((const void *)(src + qq),
                                             (__attribute__((address_space(3))) void *)(buf + qq * kWave), 16, 0, 0);
        if (c0 + kWave < jb) gnext = gids[c0 + kWave + lane < jb ? c0 + kWave + lane : jb - 1];
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_wave_barrier();
        const uint32_t cnt = jb - c0 < (uint32_t)kWave ? jb - c0 : (uint32_t)kWave;
        if (off) {
            // every record of the chunk rewritten to offsets from o
            offset_planes(buf, lane, ox, oy, oz);
            __builtin_amdgcn_wave_barrier();
            for (uint32_t s = 0; s < cnt; ++s) {
                Record a;
                a.f0 = buf[s];
                a.f1 = buf[kWave + s];
                a.f2 = buf[2 * kWave + s];
#pragma unroll
                for (uint32_t t = 0; t < R; ++t) accumulate_off_sel(a, ax[t], ay[t], az[t], T, I[t], V[t]);
            }
        } else {
            // a cell that may list a coarse Gaussian: U (p - mu)
            for (uint32_t s = 0; s < cnt; ++s) {
                Record a;
                a.f0 = buf[s];
                a.f1 = buf[kWave + s];
                a.f2 = buf[2 * kWave + s];
#pragma unroll
                for (uint32_t t = 0; t < R; ++t) accumulate_sel(a, px[t], py[t], pz[t], T, I[t], V[t]);
            }
        }
        // every lane has read the planes before the next chunk overwrites them
        __builtin_amdgcn_wave_barrier();
    }
}


__global__ __launch_bounds__(kSampBlock) void k_sample_grid(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                        const uint32_t *__restrict__ gids,
                                                        const uint32_t *__restrict__ cell_off, float T, float tau,
                                                        float *__restrict__ out_v, float *__restrict__ out_i) {
    __shared__ float4 s_grec[kSampWaves][kRecordQuads * kWave];
    const uint32_t rx = (uint32_t)(q.dims[0] / g.cells[0]);
    const uint32_t ry = (uint32_t)(q.dims[1] / g.cells[1]);
    const uint32_t rz = (uint32_t)(q.dims[2] / g.cells[2]);
    const uint32_t vpc = rx * ry * rz;
    const uint32_t wpc = (vpc + kWave - 1) / kWave;
    const uint32_t lane = threadIdx.x % kWave;
    const uint64_t wave_id =
        (uint64_t)blockIdx.x * kSampWaves + threadIdx.x / kWave;
    const uint64_t cell = wave_id / wpc;
    if (cell >= (uint64_t)g.ncells) return;
    const uint32_t chunk = (uint32_t)(wave_id - cell * wpc);
    const uint32_t local = chunk * kWave + lane;
    const uint32_t cx = (uint32_t)(cell % (uint32_t)g.cells[0]);
    const uint32_t cy = (uint32_t)((cell / (uint32_t)g.cells[0]) % (uint32_t)g.cells[1]);
    const uint32_t cz = (uint32_t)(cell / ((uint64_t)g.cells[0] * (uint32_t)g.cells[1]));
    const uint32_t lx = local % rx, ly = (local / rx) % ry, lz = local / (rx * ry);
    const int32_t vx = (int32_t)(cx * rx + lx), vy = (int32_t)(cy * ry + ly), vz = (int32_t)(cz * rz + lz);
    const float px = voxel_center(vx, g.lo[0], q.vsz[0]);
    const float py = voxel_center(vy, g.lo[1], q.vsz[1]);
    const float pz = voxel_center(vz, g.lo[2], q.vsz[2]);
    const uint32_t j0 = __builtin_amdgcn_readfirstlane(cell_off[cell]);
    const uint32_t j1 = __builtin_amdgcn_readfirstlane(cell_off[cell + 1]);
    float I = 0.0f, V = 0.0f;
    walk_staged(rec, gids, j0, j1, lane, s_grec[threadIdx.x / kWave], px, py, pz, T, I, V);
    if (local < vpc) {
        const uint64_t idx = (uint64_t)vx + (uint64_t)q.dims[0] * ((uint64_t)vy + (uint64_t)q.dims[1] * (uint64_t)vz);
        const bool def = I > tau;
        out_v[idx] = def ? V / I : 0.0f;
        out_i[idx] = def ? I : 0.0f;
    }
}

__global__ __launch_bounds__(kBlock) void k_query_keys(QueryParams q, GridParams g, uint32_t *__restrict__ keys,
                                                       uint32_t *__restrict__ ids, RadixPass0 pass0) {
    __shared__ uint32_t hist_lds[kMaxDigits];
    Pass0Hist hist(hist_lds, pass0);
#pragma unroll
    for (int it = 0; it < kSortItems; ++it) {
        const int64_t i = (int64_t)blockIdx.x * kSortTile + (int64_t)it * kBlock + threadIdx.x;
        if (i < q.n) {
            float p[3];
            bool valid;
            query_position(q, g, (uint32_t)i, p[0], p[1], p[2], valid);
            uint32_t key = kSub * (uint32_t)g.ncells;
            if (valid) {
                bool inside = true;
                int64_t c[3];
                float tx = 0.0f;
#pragma unroll
                for (int j = 0; j < 3; ++j) {
                    inside = inside && (p[j] >= g.lo[j]) && (p[j] <= g.hi[j]);
                    const float t = (p[j] - g.lo[j]) * g.invc[j];
                    int64_t ci = (int64_t)floorf(t);
                    ci = ci < 0 ? 0 : ci;
                    ci = ci > g.cells[j] - 1 ? g.cells[j] - 1 : ci;
                    c[j] = ci;
                    if (j == 0) tx = t;
                }
                if (inside) {
                    // the quarter of the cell along x: floor(4 (t - c)), exact
                    // in float32 (t - c is exact, the product by 4 too)
                    const float fq = floorf((tx - (float)c[0]) * (float)kSub);
                    const uint32_t qx = fq < 0.0f ? 0u : (fq > (float)(kSub - 1) ? kSub - 1 : (uint32_t)fq);
                    key = kSub * (uint32_t)(c[0] + (int64_t)g.cells[0] * (c[1] + (int64_t)g.cells[1] * c[2])) + qx;
                }
            }
            keys[i] = key;
            ids[i] = (uint32_t)i;
            hist.add(key);
        }
    }
    hist.finish_tile(blockIdx.x);
}

// Work items of the ordered-query sampler: one per cell holding fewer than
// 2 kDenseMin queries, one per dense item (64 or 128 queries, see
// dense_item_queries) of a denser cell. The bucket of queries outside the
// domain (key ncells) is an item with an empty list.
constexpr uint32_t kDenseMin = 32;
// A cell of at least 2 kDenseMin queries is dense: lanes are its queries,
// one or two per lane, the cell's queries split evenly over its items. Two
// a lane let each record read from LDS serve two queries (with one, the
// walk is bound by LDS reads: three 16-byte broadcast reads per candidate
// against 13 VALU operations), but make half as many items, each twice as
// long: a launch with few items per wave slot of the chip then ends with
// long items running alone. Two a lane are taken from kDenseBalance items
// per wave slot at one a lane (measured: 4.6 per slot, a 2^21-point batch
// of clustered points, runs 11 % faster with one; 218, 10^8 points, 19 %
// faster with two).
constexpr uint32_t kDenseBalance = 32;
constexpr uint32_t kChunkB = 8;  // queries evaluated together by a sparse-cell item
constexpr uint32_t kRowsMin = 4;                 // from this many queries a cell uses 4 query rows
constexpr uint32_t kRowsMax = (kDenseMin + 3) / 4;  // queries per row at most

// Work items per bucket (cell, and the outside bucket last): none for an
// empty bucket, one for a sparse one, one per dense_q queries of a dense
// one. Dense buckets' items come first in the item list, then the sparse
// buckets', each class in bucket order: items are taken in launch order,
// and the long ones started first leave no long item running alone at the
// end of the launch. The counts travel packed as (dense << 32) | sparse.
__device__ __forceinline__ uint64_t bucket_items(const uint32_t *point_off, int64_t c, int64_t nbuckets,
                                                 uint32_t dense_q) {
    if (c >= nbuckets) return 0ull;
    // the outside bucket (c = nbuckets - 1) has a single key
    const uint32_t n = point_off[c + 1 < nbuckets ? kSub * (c + 1) : kSub * c + 1] - point_off[kSub * c];
    if (n == 0) return 0ull;
    if (n < 2 * kDenseMin) return 1ull;
    return (uint64_t)((n + dense_q - 1) / dense_q) << 32;
}

// Buckets are taken kItemGroup at a time (kItemsPerThread per thread).
constexpr int kItemsPerThread = 4;
constexpr int kItemGroup = kBlock * kItemsPerThread;  // 1024
// Up to this many groups, the offsets kernel sums the other groups itself;
// beyond, their sums are scanned by a separate pass (which also writes the
// total after them).
constexpr int64_t kInlineGroups = 1024;

__global__ __launch_bounds__(kBlock) void k_item_sums(const uint32_t *__restrict__ point_off, int64_t nbuckets,
                                                      uint32_t dense_q, uint64_t *__restrict__ group_sum) {
    __shared__ uint64_t lds[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kItemGroup + (int64_t)threadIdx.x * kItemsPerThread;
    uint64_t s = 0;
#pragma unroll
    for (int i = 0; i < kItemsPerThread; ++i) s += bucket_items(point_off, base + i, nbuckets, dense_q);
    uint64_t tot;
    (void)block_excl_scan(s, lds, &tot);
    if (threadIdx.x == 0) group_sum[blockIdx.x] = tot;
}

// item_off[c] for c <= nbuckets: the first item of bucket c (item_off[nbuckets]
// = the total), and the item list: item_off[c] .. item_off[c] + items(c) - 1
// name bucket c. group_sum: the groups' sums, or (scanned) their exclusive
// prefixes followed by the total.
__global__ __launch_bounds__(kBlock) void k_item_offsets(const uint32_t *__restrict__ point_off, int64_t nbuckets,
                                                         uint32_t dense_q, const uint64_t *__restrict__ group_sum,
                                                         int64_t ngroups,
                                                         bool scanned, uint32_t *__restrict__ item_off,
                                                         uint32_t *__restrict__ items, int64_t max_items) {
    __shared__ uint64_t lds[kWavesPerBlock];
    uint64_t prefix, total;
    if (scanned) {
        prefix = group_sum[blockIdx.x];
        total = group_sum[ngroups];
    } else {
        uint64_t p = 0, a = 0;
        for (uint32_t j = threadIdx.x; j < (uint32_t)ngroups; j += kBlock) {
            const uint64_t v = group_sum[j];
            a += v;
            if (j < blockIdx.x) p += v;
        }
        uint64_t t;
        (void)block_excl_scan(p, lds, &t);
        prefix = t;
        (void)block_excl_scan(a, lds, &t);
        total = t;
    }
    const uint32_t dense_total = (uint32_t)(total >> 32);
    const int64_t base = (int64_t)blockIdx.x * kItemGroup + (int64_t)threadIdx.x * kItemsPerThread;
    uint64_t v[kItemsPerThread];
    uint64_t s = 0;
#pragma unroll
    for (int i = 0; i < kItemsPerThread; ++i) {
        v[i] = bucket_items(point_off, base + i, nbuckets, dense_q);
        s += v[i];
    }
    uint64_t tot;
    uint64_t run = block_excl_scan(s, lds, &tot) + prefix;
#pragma unroll
    for (int i = 0; i < kItemsPerThread; ++i) {
        const int64_t c = base + i;
        const bool dense = (v[i] >> 32) != 0;
        const uint32_t first = dense ? (uint32_t)(run >> 32) : dense_total + (uint32_t)run;
        const uint32_t cnt = dense ? (uint32_t)(v[i] >> 32) : (uint32_t)v[i];
        if (c < nbuckets) item_off[c] = first;
        if (c == nbuckets) item_off[c] = dense_total + (uint32_t)total;
        for (uint32_t k = 0; k < cnt; ++k)
            if ((int64_t)(first + k) < max_items) items[first + k] = (uint32_t)c;
        run += v[i];
    }
}

// G of a record at a point, 0 past the cutoff.
__device__ __forceinline__ float eval_g(const Record &r, float px, float py, float pz, float T) {
    const float Q = cutoff_q(r, px, py, pz);
    return Q <= T ? exp2_hw(-Q) : 0.0f;
}

// sum over the 64 lanes, returned to every lane
__device__ __forceinline__ float wave_total(float x) {
    const float r = row16_sum(x);
    return (readlane_f(r, 0) + readlane_f(r, 16)) + (readlane_f(r, 32) + readlane_f(r, 48));
}

// Outputs of one query: (Phi, I) at its id in query order, and its position
// and (Phi, I) at its index k in plan order for the backward.
__device__ __forceinline__ void write_out(float I, float V, float tau, bool work, uint32_t pid, uint32_t k, float px,
                                          float py, float pz, float *out_v, float *out_i, const PlanResults &pr) {
    const bool def = work && I > tau;
    const float phi = def ? V / I : 0.0f, inf = def ? I : 0.0f;
    out_v[pid] = phi;
    out_i[pid] = inf;
    pr.pos[k] = make_float4(px, py, pz, 0.0f);
    pr.out[k] = make_float2(phi, inf);
}

// Sum over the SL lanes of a candidate-slot row (16: DPP row sum; 8: quad
// sums, then row_half_mirror pairs the two quads of each half row).
template <uint32_t SL>
__device__ __forceinline__ float slot_sum(float x) {
    if (SL == 16) return row16_sum(x);
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x141>(x);
    return x;
}

// ROWS query rows x (64 / ROWS) candidate slots for a cell of
// n < 8 ROWS queries: lane (r, s) evaluates queries r, r + ROWS, ... against
// candidates s, s + 64 / ROWS, ... of the list; a query's partial sums are
// then summed over its row with DPP.
template <uint32_t ROWS>
__device__ __forceinline__ void query_rows(uint32_t lane, uint32_t n, uint32_t pa, uint32_t ja, uint32_t jb,
                                           uint32_t c, uint32_t ncells, const QueryParams &q, const GridParams &g,
                                           const Record *__restrict__ rec, const uint32_t *__restrict__ gids,
                                           const uint32_t *__restrict__ order, float T, float tau,
                                           float *__restrict__ out_v, float *__restrict__ out_i,
                                           const PlanResults &pr, float4 *buf) {
        constexpr uint32_t SL = kWave / ROWS;  // candidate slots per row
        const uint32_t row = lane / SL, sl = lane % SL;
        const uint32_t nt = (n + ROWS - 1) / ROWS;  // queries per row, <= kRowsMax
        uint32_t pid = 0;
        float mx = 0.0f, my = 0.0f, mz = 0.0f;
        bool valid = false;
        if (lane < n) {
            pid = order[pa + lane];
            if ((int64_t)pid < q.n) query_position(q, g, pid, mx, my, mz, valid);
        }
        float px[kRowsMax], py[kRowsMax], pz[kRowsMax], Ip[kRowsMax], Vp[kRowsMax];
#pragma unroll
        for (uint32_t t = 0; t < kRowsMax; ++t) {
            px[t] = py[t] = pz[t] = 0.0f;
            Ip[t] = Vp[t] = 0.0f;
            if (t < nt) {
                const int src = (int)(row + ROWS * t);
                px[t] = __shfl(mx, src, 64);
                py[t] = __shfl(my, src, 64);
                pz[t] = __shfl(mz, src, 64);
            }
        }
        // The list is taken 64 candidates at a time: lane l copies candidate
        // c0 + l's record from memory straight into the wave's LDS planes
        // (lanes past the list copy its last record), the ids of the next 64
        // are fetched meanwhile, and the steps of SL read the records from
        // LDS, so a chunk waits for memory once instead of once per step.
        uint32_t gnext = 0;
        if (ja < jb) gnext = gids[ja + lane < jb ? ja + lane : jb - 1];
        for (uint32_t c0 = ja; c0 < jb; c0 += kWave) {
            const float4 *src = (const float4 *)(rec + gnext);
#pragma unroll
            for (int qq = 0; qq < kRecordQuads; ++qq)
                __builtin_amdgcn_global_load_lds((const void *)(src + qq),
                                                 (__attribute__((address_space(3))) void *)(buf + qq * kWave), 16, 0, 0);
            if (c0 + kWave < jb) gnext = gids[c0 + kWave + lane < jb ? c0 + kWave + lane : jb - 1];
            __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_wave_barrier();
            const uint32_t left = jb - c0;
            const uint32_t nstep = left >= (uint32_t)kWave ? kWave / SL : (left + SL - 1) / SL;
            for (uint32_t st = 0; st < nstep; ++st) {
                const uint32_t sidx = SL * st + sl;
                Record r;
                r.f0 = buf[sidx];
                r.f1 = buf[kWave + sidx];
                r.f2 = buf[2 * kWave + sidx];
                if (c0 + sidx >= jb) r.f0.w = r.f1.w = 0.0f;  // past the list: weight 0
#pragma unroll
                for (uint32_t t = 0; t < kRowsMax; ++t) {
                    if (t < nt) {
                        const float G = eval_g(r, px[t], py[t], pz[t], T);
                        Ip[t] = fmaf_(r.f0.w, G, Ip[t]);
                        Vp[t] = fmaf_(r.f1.w, G, Vp[t]);
                    }
                }
            }
            // every lane has read the planes before the next chunk overwrites them
            __builtin_amdgcn_wave_barrier();
        }
        float Io = 0.0f, Vo = 0.0f;
#pragma unroll
        for (uint32_t t = 0; t < kRowsMax; ++t) {
            if (t < nt) {
                const float It = slot_sum<SL>(Ip[t]), Vt = slot_sum<SL>(Vp[t]);
                if (sl == t) {
                    Io = It;
                    Vo = Vt;
                }
            }
        }
        // lane (r, t) writes query r + ROWS t, whose id and position that lane holds
        const uint32_t qi = row + ROWS * sl;
        const int src = (int)(qi & 63u);
        const uint32_t wpid = __shfl(pid, src, 64);
        const float wx = __shfl(mx, src, 64), wy = __shfl(my, src, 64), wz = __shfl(mz, src, 64);
        const bool wvalid = __shfl((int)valid, src, 64) != 0;
        if (sl < nt && qi < n && (int64_t)wpid < q.n)
            write_out(Io, Vo, tau, wvalid && c < ncells, wpid, pa + qi, wx, wy, wz, out_v, out_i, pr);
}

// A dense cell's work item: queries [qa, qa + qn) of the plan, qn <= 64 R;
// lane l takes queries qa + l + 64 t, t < R.
template <uint32_t R>
__device__ __forceinline__ void dense_item(uint32_t lane, uint32_t qa, uint32_t qn, uint32_t ja,
                                           uint32_t jb, uint32_t c, uint32_t ncells, const QueryParams &q,
                                           const GridParams &g, const Record *__restrict__ rec,
                                           bool off, const uint32_t *__restrict__ gids,
                                           const uint32_t *__restrict__ order, float T, float tau,
                                           float *__restrict__ out_v, float *__restrict__ out_i,
                                           const PlanResults &pr, float4 *buf) {
    float px[R], py[R], pz[R], I[R], V[R];
    uint32_t pid[R];
    bool valid[R];
#pragma unroll
    for (uint32_t t = 0; t < R; ++t) {
        px[t] = py[t] = pz[t] = 0.0f;
        I[t] = V[t] = 0.0f;
        pid[t] = 0xFFFFFFFFu;
        valid[t] = false;
        if (lane + kWave * t < qn) {
            pid[t] = order[qa + lane + kWave * t];
            if ((int64_t)pid[t] < q.n) query_position(q, g, pid[t], px[t], py[t], pz[t], valid[t]);
        }
    }
    float ox = 0.0f, oy = 0.0f, oz = 0.0f;
    if (c < ncells) cell_centre(g, c, ox, oy, oz);
    walk_staged_r<R>(rec, off, gids, ja, jb, lane, buf, px, py, pz, ox, oy, oz, T, I, V);
#pragma unroll
    for (uint32_t t = 0; t < R; ++t)
        if (lane + kWave * t < qn && (int64_t)pid[t] < q.n)
            write_out(I[t], V[t], tau, valid[t] && c < ncells, pid[t], qa + lane + kWave * t, px[t], py[t], pz[t],
                      out_v, out_i, pr);
}

// One wavefront per item, by the queries n of the cell:
//  * n >= 64: lanes are queries, up to dense_q / 64 each (dense_q
//    queries per item, a cell's queries split evenly over its items), and
//    walk the list together, the records staged in LDS;
//  * 4 <= n < 64: query rows x candidate slots (4 x 16 below 32 queries,
//    8 x 8 from 32), records staged in LDS 64 at a time;
//  * n < 4: lanes are the cell's candidates (64 at a time) and the queries
//    are visited in turn, their positions broadcast from SGPRs.
// Every query's sums are reduced in a fixed order.
// Seven waves per SIMD (at most 72 VGPRs, which the row layouts' per-row
// arrays need; eight would spill them to scratch).
__global__ __launch_bounds__(kSampBlock, kSampPerSimd) void k_sample_cells(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                         const uint8_t *__restrict__ cell_coarse,
                                                         const uint32_t *__restrict__ gids,
                                                         const uint32_t *__restrict__ cell_off,
                                                         const uint32_t *__restrict__ point_off,
                                                         const uint32_t *__restrict__ order,
                                                         const uint32_t *__restrict__ item_off,
                                                         const uint32_t *__restrict__ items, int64_t max_items,
                                                         uint32_t dense_q, float T, float tau,
                                                         float *__restrict__ out_v, float *__restrict__ out_i,
                                                         PlanResults pr) {
    // per wave: the records of 64 candidates, as three 1 KiB planes of
    // 16-byte quarters (quarter q of candidate s at [q][s])
    __shared__ float4 s_rec[kSampWaves][kRecordQuads * kWave];
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t ncells = (uint32_t)g.ncells;
    const uint32_t bid = xcd_group<kXcdItems>(blockIdx.x, gridDim.x);
    const uint64_t w = (uint64_t)bid * kSampWaves + threadIdx.x / kWave;
    const uint32_t tot = ((ConstU32 *)item_off)[ncells + 1];
    const uint64_t total = tot < (uint64_t)max_items ? tot : (uint64_t)max_items;
    if (w >= total) return;
    const uint32_t c = __builtin_amdgcn_readfirstlane(((ConstU32 *)items)[w]);
    const uint32_t chunk = (uint32_t)w - ((ConstU32 *)item_off)[c];
    const uint32_t pa = ((ConstU32 *)point_off)[kSub * c];
    const uint32_t pb = ((ConstU32 *)point_off)[c < ncells ? kSub * (c + 1) : kSub * c + 1];
    const uint32_t n = pb - pa;
    uint32_t ja = 0, jb = 0;
    if (c < ncells) {
        ja = ((ConstU32 *)cell_off)[c];
        jb = ((ConstU32 *)cell_off)[c + 1];
    }
    if (n >= 2 * kDenseMin) {
        // offsets from the cell's centre unless the cell may list a Gaussian
        // too small for them (see offset_planes)
        const bool off = c >= ncells || __builtin_amdgcn_readfirstlane(cell_coarse[c]) == 0;
        const uint32_t nit = (n + dense_q - 1) / dense_q;
        const uint32_t per = (n + nit - 1) / nit;
        const uint32_t qa = pa + chunk * per;
        const uint32_t qn = pb - qa < per ? pb - qa : per;
        float4 *buf = s_rec[threadIdx.x / kWave];
        if (qn <= (uint32_t)kWave)
            dense_item<1>(lane, qa, qn, ja, jb, c, ncells, q, g, rec, off, gids, order, T, tau, out_v, out_i, pr,
                          buf);
        else
            dense_item<2>(lane, qa, qn, ja, jb, c, ncells, q, g, rec, off, gids, order, T, tau, out_v, out_i, pr,
                          buf);
        return;
    }
    if (n >= kRowsMin) {
        float4 *buf = s_rec[threadIdx.x / kWave];
        if (n >= kDenseMin)
            query_rows<8>(lane, n, pa, ja, jb, c, ncells, q, g, rec, gids, order, T, tau, out_v, out_i, pr, buf);
        else
            query_rows<4>(lane, n, pa, ja, jb, c, ncells, q, g, rec, gids, order, T, tau, out_v, out_i, pr, buf);
        return;
    }
    for (uint32_t p0 = pa; p0 < pb; p0 += kChunkB) {
        const uint32_t m = (pb - p0) < kChunkB ? (pb - p0) : kChunkB;
        uint32_t pid = 0;
        float mx = 0.0f, my = 0.0f, mz = 0.0f;
        bool valid = false;
        if (lane < m) {
            pid = order[p0 + lane];
            if ((int64_t)pid < q.n) query_position(q, g, pid, mx, my, mz, valid);
        }
        float Ip[kChunkB], Vp[kChunkB];
#pragma unroll
        for (uint32_t t = 0; t < kChunkB; ++t) Ip[t] = Vp[t] = 0.0f;
        for (uint32_t j0 = ja; j0 < jb; j0 += kWave) {
            const uint32_t j = j0 + lane;
            Record r;
            if (j < jb) {
                r = rec[gids[j]];
            } else {
                r.f0 = r.f1 = r.f2 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
#pragma unroll
            for (uint32_t t = 0; t < kChunkB; ++t) {
                if (t < m) {
                    const float G = eval_g(r, readlane_f(mx, t), readlane_f(my, t), readlane_f(mz, t), T);
                    Ip[t] = fmaf_(r.f0.w, G, Ip[t]);
                    Vp[t] = fmaf_(r.f1.w, G, Vp[t]);
                }
            }
        }
        float Io = 0.0f, Vo = 0.0f;
#pragma unroll
        for (uint32_t t = 0; t < kChunkB; ++t) {
            if (t < m) {
                const float It = wave_total(Ip[t]), Vt = wave_total(Vp[t]);
                if (lane == t) {
                    Io = It;
                    Vo = Vt;
                }
            }
        }
        if (lane < m && (int64_t)pid < q.n)
            write_out(Io, Vo, tau, valid && c < ncells, pid, p0 + lane, mx, my, mz, out_v, out_i, pr);
    }
}

// Pairs the forward tests and the pairs among them that pass the cutoff,
// for measurement: thread t takes query t of the grid (x fastest) or the
// t-th query in plan order, walks its cell's list with the samplers' own
// float32 test and counts. Summed per block, then into totals[0] (tests)
// and totals[1] (passing) with one integer atomic each per block (the sums
// do not depend on their order).
__global__ __launch_bounds__(kBlock) void k_count_sample_pairs(QueryParams q, GridParams g,
                                                               const Record *__restrict__ rec,
                                                               const uint32_t *__restrict__ gids,
                                                               const uint32_t *__restrict__ cell_off,
                                                               const uint32_t *__restrict__ plan_keys,
                                                               const float4 *__restrict__ plan_pos, float T,
                                                               unsigned long long *totals) {
    __shared__ unsigned long long lds[2][kWavesPerBlock];
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    unsigned long long tests = 0, hits = 0;
    if (t < q.n) {
        int64_t c = -1;
        float px = 0.0f, py = 0.0f, pz = 0.0f;
        if (q.kind == 0) {
            const uint32_t nx = (uint32_t)q.dims[0], ny = (uint32_t)q.dims[1];
            const uint32_t vx = (uint32_t)(t % nx), vy = (uint32_t)((t / nx) % ny), vz = (uint32_t)(t / ((int64_t)nx * ny));
            const uint32_t rx = nx / (uint32_t)g.cells[0], ry = ny / (uint32_t)g.cells[1];
            const uint32_t rz = (uint32_t)q.dims[2] / (uint32_t)g.cells[2];
            c = (int64_t)(vx / rx) + (int64_t)g.cells[0] * ((int64_t)(vy / ry) + (int64_t)g.cells[1] * (vz / rz));
            px = voxel_center((int32_t)vx, g.lo[0], q.vsz[0]);
            py = voxel_center((int32_t)vy, g.lo[1], q.vsz[1]);
            pz = voxel_center((int32_t)vz, g.lo[2], q.vsz[2]);
        } else {
            const uint32_t cc = plan_keys[t] / kSub;
            if ((int64_t)cc < g.ncells) {
                c = cc;
                const float4 p = plan_pos[t];
                px = p.x;
                py = p.y;
                pz = p.z;
            }
        }
        if (c >= 0) {
            const uint32_t j0 = cell_off[c], j1 = cell_off[c + 1];
            tests = j1 - j0;
            for (uint32_t j = j0; j < j1; ++j) hits += cutoff_q(rec[gids[j]], px, py, pz) <= T ? 1u : 0u;
        }
    }
    const uint32_t lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        tests += __shfl_xor(tests, o, kWave);
        hits += __shfl_xor(hits, o, kWave);
    }
    if (lane == 0) {
        lds[0][wid] = tests;
        lds[1][wid] = hits;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        unsigned long long s = 0;
        for (int w = 0; w < kWavesPerBlock; ++w) s += lds[threadIdx.x][w];
        if (s) atomicAdd(totals + threadIdx.x, s);
    }
}

}  // namespace

hipError_t launch_count_sample_pairs(const QueryParams &q, const GridParams &g, const Record *rec,
                                     const uint32_t *gids, const uint32_t *cell_off, const uint32_t *plan_keys,
                                     const float4 *plan_pos, float T, unsigned long long *totals, hipStream_t s) {
    hipError_t e = fill_u32((uint32_t *)totals, 0u, 4, s);
    if (e != hipSuccess || q.n <= 0) return e;
    hipLaunchKernelGGL(k_count_sample_pairs, dim3((uint32_t)((q.n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, q, g,
                       rec, gids, cell_off, plan_keys, plan_pos, T, totals);
    return hipGetLastError();
}

hipError_t launch_query_keys(const QueryParams &q, const GridParams &g, uint32_t *keys, uint32_t *ids,
                             const RadixPass0 &pass0, hipStream_t s) {
    if (q.n <= 0) return hipSuccess;
    prof_begin("query_keys", s);
    hipLaunchKernelGGL(k_query_keys, dim3((uint32_t)((q.n + kSortTile - 1) / kSortTile)), dim3(kBlock), 0, s, q, g,
                       keys, ids, pass0);
    prof_end("query_keys", s);
    return hipGetLastError();
}

hipError_t launch_sample_grid(const QueryParams &q, const GridParams &g, const Record *rec, const uint32_t *gids,
                              const uint32_t *cell_off, float T, float tau, float *out_v, float *out_i,
                              hipStream_t s) {
    const int64_t vpc = (int64_t)(q.dims[0] / g.cells[0]) * (q.dims[1] / g.cells[1]) * (q.dims[2] / g.cells[2]);
    const int64_t wpc = (vpc + kWave - 1) / kWave;
    const int64_t waves = g.ncells * wpc;
    const int64_t blocks = (waves + kSampWaves - 1) / kSampWaves;
    if (blocks <= 0) return hipSuccess;
    prof_begin("sample_grid", s);
    hipLaunchKernelGGL(k_sample_grid, dim3((uint32_t)blocks), dim3(kSampBlock), 0, s, q, g, rec, gids, cell_off, T, tau,
                       out_v, out_i);
    prof_end("sample_grid", s);
    return hipGetLastError();
}

// Queries per dense work item for nq ordered queries on the current device:
// 128 (two a lane) from kDenseBalance items per wave slot of the chip at
// 64, else 64. The item list and the sampler both take it from nq, so they
// agree.
static uint32_t dense_item_queries(int64_t nq) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
        (void)hipGetLastError();
        cus = 256;
    }
    const int64_t slots = (int64_t)cus * 4 * kSampPerSimd;  // 4 SIMDs a CU
    return nq / kWave >= (int64_t)kDenseBalance * slots ? 2u * kWave : (uint32_t)kWave;
}

hipError_t launch_cell_items(int64_t nq, const GridParams &g, const uint32_t *point_off, const PointItems &it,
                             hipStream_t s) {
    if (nq <= 0) return hipSuccess;
    const uint32_t dense_q = dense_item_queries(nq);
    const int64_t nbuckets = g.ncells + 1;  // cells and the outside bucket
    // buckets 0..nbuckets-1 and one empty element after them (its offset is the total)
    const int64_t ngroups = (nbuckets + 1 + kItemGroup - 1) / kItemGroup;
    const bool scanned = ngroups > kInlineGroups;
    prof_begin("cell_items", s);
    hipLaunchKernelGGL(k_item_sums, dim3((uint32_t)ngroups), dim3(kBlock), 0, s, point_off, nbuckets, dense_q,
                       it.group_sum);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && scanned)
        e = exclusive_scan_u64_total(it.group_sum, it.group_sum, ngroups, it.group_sum + ngroups, it.scan_work, s);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_item_offsets, dim3((uint32_t)ngroups), dim3(kBlock), 0, s, point_off, nbuckets,
                           dense_q, it.group_sum, ngroups, scanned, it.item_off, it.items, it.max_items);
        e = hipGetLastError();
    }
    prof_end("cell_items", s);
    return e;
}

hipError_t launch_sample_points(const QueryParams &q, const GridParams &g, const Record *rec, const uint8_t *cell_coarse,
                                const uint32_t *gids, const uint32_t *cell_off, const uint32_t *order, const uint32_t *point_off,
                                const PointItems &it, float T, float tau, float *out_v, float *out_i,
                                const PlanResults &pr, hipStream_t s) {
    if (q.n <= 0) return hipSuccess;
    prof_begin("sample_points", s);
    hipLaunchKernelGGL(k_sample_cells, dim3((uint32_t)((it.max_items + kSampWaves - 1) / kSampWaves)),
                       dim3(kSampBlock), 0, s, q, g, rec, cell_coarse, gids, cell_off, point_off, order, it.item_off,
                       it.items,
                       it.max_items, dense_item_queries(q.n), T, tau, out_v, out_i, pr);
    prof_end("sample_points", s);
    return hipGetLastError();
}

}  // namespace gs
