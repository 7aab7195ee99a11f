// Cell index of the Gaussians (paper Sec. 4.1.1 and Sec. 4.1.2):
//  - preprocess: per Gaussian, the axis-aligned box of its cutoff ellipsoid
//    in cells (canonical float32, each operation rounded separately), its
//    cell count, and the evaluation record used by the samplers;
//  - emit: one (cell key, Gaussian id) pair per cell of every box,
//    parallel over pairs with a per-tile load-balanced search for the owning
//    Gaussian (the paper parallelises this step over intersections for the
//    same reason: box sizes vary by orders of magnitude in 3D).
// The pairs are then sorted by key (primitives.hip) and the per-cell ranges
// taken from the sorted keys.
#include "expand.h"
#include "internal.h"
#include "radix.h"

#pragma clang fp contract(off)

namespace gs {

namespace {

__device__ __forceinline__ bool finite_f(float x) { return __builtin_isfinite(x); }

__global__ __launch_bounds__(kBlock) void k_preprocess(const float *__restrict__ mean, const float *__restrict__ scale,
                                                       const float *__restrict__ rot, const float *__restrict__ value,
                                                       const float *__restrict__ weight, int64_t n, GridParams g,
                                                       float rci, Record *__restrict__ rec, CellBox *__restrict__ box,
                                                       uint64_t *__restrict__ count) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == n) count[n] = 0;
    if (i >= n) return;
    const float mu[3] = {mean[3 * i], mean[3 * i + 1], mean[3 * i + 2]};
    const float s[3] = {scale[3 * i], scale[3 * i + 1], scale[3 * i + 2]};
    const float q[4] = {rot[4 * i], rot[4 * i + 1], rot[4 * i + 2], rot[4 * i + 3]};
    const float v = value[i], w = weight[i];

    bool valid = finite_f(v) && finite_f(w);
#pragma unroll
    for (int j = 0; j < 3; ++j) valid = valid && finite_f(mu[j]) && finite_f(s[j]) && (s[j] > 0.0f);
#pragma unroll
    for (int j = 0; j < 4; ++j) valid = valid && finite_f(q[j]);

    // canonical float32 rotation (every product and sum rounded in this order)
    const float n2 = ((q[0] * q[0] + q[1] * q[1]) + q[2] * q[2]) + q[3] * q[3];
    valid = valid && (n2 > 0.0f) && finite_f(n2);
    const float inv = 1.0f / sqrtf(n2);
    const float qw = q[0] * inv, qx = q[1] * inv, qy = q[2] * inv, qz = q[3] * inv;
    float R[3][3];
    R[0][0] = 1.0f - 2.0f * (qy * qy + qz * qz);
    R[0][1] = 2.0f * (qx * qy - qw * qz);
    R[0][2] = 2.0f * (qx * qz + qw * qy);
    R[1][0] = 2.0f * (qx * qy + qw * qz);
    R[1][1] = 1.0f - 2.0f * (qx * qx + qz * qz);
    R[1][2] = 2.0f * (qy * qz - qw * qx);
    R[2][0] = 2.0f * (qx * qz - qw * qy);
    R[2][1] = 2.0f * (qy * qz + qw * qx);
    R[2][2] = 1.0f - 2.0f * (qx * qx + qy * qy);

    int lo_c[3], hi_c[3];
    uint64_t cnt = 1;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const float a0 = R[j][0] * s[0], a1 = R[j][1] * s[1], a2 = R[j][2] * s[2];
        const float var = (a0 * a0 + a1 * a1) + a2 * a2;
        const float h = rci * sqrtf(var);
        const float lo = mu[j] - h, hi = mu[j] + h;
        const float tl = (lo - g.lo[j]) * g.invc[j];
        const float th = (hi - g.lo[j]) * g.invc[j];
        const float fl = floorf(tl), fh = floorf(th);
        const float cmax = (float)(g.cells[j] - 1);
        if (!finite_f(h) || !finite_f(fl) || !finite_f(fh) || !(fh >= 0.0f) || !(fl <= cmax)) valid = false;
        lo_c[j] = valid ? (int)(fl > 0.0f ? fl : 0.0f) : 0;
        hi_c[j] = valid ? (int)(fh < cmax ? fh : cmax) : -1;
        cnt *= valid ? (uint64_t)(hi_c[j] - lo_c[j] + 1) : 0ull;
    }
    if (!valid) {
        lo_c[0] = lo_c[1] = lo_c[2] = 0;
        hi_c[0] = hi_c[1] = hi_c[2] = -1;
        cnt = 0;
    }
    count[i] = cnt;
    CellBox b;
    b.lo = make_int4(lo_c[0], lo_c[1], lo_c[2], 0);
    b.hi = make_int4(hi_c[0], hi_c[1], hi_c[2], 0);
    box[i] = b;

    // evaluation record: M = S^-1 R^T formed in float64, rounded once
    Record r;
    if (valid) {
        const double qn = sqrt((double)q[0] * q[0] + (double)q[1] * q[1] + (double)q[2] * q[2] + (double)q[3] * q[3]);
        const double w_ = q[0] / qn, x = q[1] / qn, y = q[2] / qn, z = q[3] / qn;
        double Rd[3][3];
        Rd[0][0] = 1.0 - 2.0 * (y * y + z * z);
        Rd[0][1] = 2.0 * (x * y - w_ * z);
        Rd[0][2] = 2.0 * (x * z + w_ * y);
        Rd[1][0] = 2.0 * (x * y + w_ * z);
        Rd[1][1] = 1.0 - 2.0 * (x * x + z * z);
        Rd[1][2] = 2.0 * (y * z - w_ * x);
        Rd[2][0] = 2.0 * (x * z - w_ * y);
        Rd[2][1] = 2.0 * (y * z + w_ * x);
        Rd[2][2] = 1.0 - 2.0 * (x * x + y * y);
        float M[3][3];
#pragma unroll
        for (int k = 0; k < 3; ++k)
#pragma unroll
            for (int j = 0; j < 3; ++j) M[k][j] = (float)(Rd[j][k] / (double)s[k]);
        r.r0 = make_float4(mu[0], mu[1], mu[2], w);
        r.r1 = make_float4(M[0][0], M[0][1], M[0][2], v);
        r.r2 = make_float4(M[1][0], M[1][1], M[1][2], 0.0f);
        r.r3 = make_float4(M[2][0], M[2][1], M[2][2], 0.0f);
    } else {
        r.r0 = r.r1 = r.r2 = r.r3 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    rec[i] = r;
}

__global__ __launch_bounds__(kBlock) void k_emit(const uint64_t *__restrict__ pair_off,
                                                 const CellBox *__restrict__ box, int64_t n, int64_t npairs,
                                                 const uint32_t *__restrict__ tile_first, GridParams g,
                                                 uint32_t *__restrict__ keys, uint32_t *__restrict__ gids,
                                                 RadixPass0 pass0) {
    __shared__ uint32_t head[kExpandTile];
    __shared__ uint32_t wmax[kWavesPerBlock];
    __shared__ uint32_t hist_lds[kMaxDigits];
    Pass0Hist hist(hist_lds, pass0);
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const uint32_t tile = xcd_block(blockIdx.x, gridDim.x);
    const uint64_t tile_begin = (uint64_t)tile * kExpandTile;
    const uint64_t rem = (uint64_t)npairs - tile_begin;
    const uint32_t tile_cnt = rem < (uint64_t)kExpandTile ? (uint32_t)rem : (uint32_t)kExpandTile;
    const int64_t gfirst = tile_first[tile];
    const int64_t glast = (tile + 1 < gridDim.x) ? (int64_t)tile_first[tile + 1] : n - 1;
    for (uint32_t s = tid; s < (uint32_t)kExpandTile; s += kBlock) head[s] = 0;
    __syncthreads();
    // mark the first pair of every Gaussian that starts inside the tile
    for (int64_t gg = gfirst + 1 + tid; gg <= glast; gg += kBlock) {
        const uint64_t pos = pair_off[gg] - tile_begin;
        if (pos < tile_cnt) atomicMax(&head[pos], (uint32_t)(gg - gfirst));
    }
    __syncthreads();
    // inclusive max-scan carries each mark over the Gaussian's pairs
    uint32_t run = 0;
    const uint32_t b0 = tid * kExpandItems;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t h = head[b0 + i];
        run = h > run ? h : run;
        head[b0 + i] = run;
    }
    const uint32_t incl = wave_incl_max(run);
    uint32_t excl = __shfl_up(incl, 1, 64);
    if (lane == 0) excl = 0;
    if (lane == kWave - 1) wmax[wave] = incl;
    __syncthreads();
    uint32_t wpre = 0;
    for (uint32_t w = 0; w < wave; ++w) wpre = wmax[w] > wpre ? wmax[w] : wpre;
    const uint32_t carry = excl > wpre ? excl : wpre;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t h = head[b0 + i];
        head[b0 + i] = h > carry ? h : carry;
    }
    __syncthreads();
    const int64_t Cx = g.cells[0], Cy = g.cells[1];
#pragma unroll 2
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t slot = (uint32_t)i * kBlock + tid;
        if (slot < tile_cnt) {
            const int64_t gg = gfirst + head[slot];
            const uint32_t local = (uint32_t)(tile_begin + slot - pair_off[gg]);
            const CellBox b = box[gg];
            const uint32_t nx = (uint32_t)(b.hi.x - b.lo.x + 1), ny = (uint32_t)(b.hi.y - b.lo.y + 1);
            const uint32_t t = local / nx;
            const int64_t cx = b.lo.x + (int64_t)(local - t * nx);
            const int64_t cy = b.lo.y + (int64_t)(t % ny);
            const int64_t cz = b.lo.z + (int64_t)(t / ny);
            const uint32_t key = (uint32_t)(cx + Cx * (cy + Cy * cz));
            keys[tile_begin + slot] = key;
            gids[tile_begin + slot] = (uint32_t)gg;
            hist.add(key);
        }
    }
    hist.finish_tile(tile);
}

// Sort key of each Gaussian for the spatial visiting order: the cell key of
// its box's low corner (ncells for an empty box), shifted right by `shift`
// so that one radix pass orders it. Tiles of kSortTile Gaussians per
// workgroup, with the pass's digit counts.
__global__ __launch_bounds__(kBlock) void k_gauss_keys(const CellBox *__restrict__ box, int64_t n, GridParams g,
                                                       int shift, uint32_t *__restrict__ keys,
                                                       uint32_t *__restrict__ ids, RadixPass0 pass0) {
    __shared__ uint32_t hist_lds[kMaxDigits];
    Pass0Hist hist(hist_lds, pass0);
#pragma unroll
    for (int it = 0; it < kSortItems; ++it) {
        const int64_t i = (int64_t)blockIdx.x * kSortTile + (int64_t)it * kBlock + threadIdx.x;
        if (i < n) {
            const CellBox b = box[i];
            uint32_t key = (uint32_t)g.ncells;
            if (b.hi.x >= b.lo.x)
                key = (uint32_t)((int64_t)b.lo.x + (int64_t)g.cells[0] * ((int64_t)b.lo.y + (int64_t)g.cells[1] * b.lo.z));
            key >>= shift;
            keys[i] = key;
            ids[i] = (uint32_t)i;
            hist.add(key);
        }
    }
    hist.finish_tile(blockIdx.x);
}

// First segment of every emit tile: tile_first[t] = the Gaussian owning pair
// t * kSortTile (all searches run in parallel, one thread per tile).
__global__ __launch_bounds__(kBlock) void k_tile_first(const uint64_t *__restrict__ pair_off, int64_t n,
                                                       int64_t npairs, uint32_t ntiles,
                                                       uint32_t *__restrict__ tile_first) {
    const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= ntiles) return;
    tile_first[t] = (uint32_t)segment_search(pair_off, n, (uint64_t)t * kSortTile);
}

}  // namespace

hipError_t launch_gauss_keys(const CellBox *box, int64_t n, const GridParams &g, int shift, uint32_t *keys,
                             uint32_t *ids, const RadixPass0 &pass0, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    prof_begin("gauss_keys", s);
    hipLaunchKernelGGL(k_gauss_keys, dim3((uint32_t)((n + kSortTile - 1) / kSortTile)), dim3(kBlock), 0, s, box, n, g,
                       shift, keys, ids, pass0);
    prof_end("gauss_keys", s);
    return hipGetLastError();
}

hipError_t launch_preprocess(const float *mean, const float *scale, const float *rot, const float *value,
                             const float *weight, int64_t n, const GridParams &g, float rci, Record *rec,
                             CellBox *box, uint64_t *count, hipStream_t s) {
    const int64_t threads = n + 1;
    const uint32_t blocks = (uint32_t)((threads + kBlock - 1) / kBlock);
    prof_begin("preprocess", s);
    hipLaunchKernelGGL(k_preprocess, dim3(blocks), dim3(kBlock), 0, s, mean, scale, rot, value, weight, n, g, rci, rec,
                       box, count);
    prof_end("preprocess", s);
    return hipGetLastError();
}

hipError_t launch_emit(const uint64_t *pair_off, const CellBox *box, int64_t n, int64_t npairs, const GridParams &g,
                       uint32_t *tile_first, uint32_t *keys, uint32_t *gids, const RadixPass0 &pass0, hipStream_t s) {
    if (npairs <= 0 || n <= 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((npairs + kExpandTile - 1) / kExpandTile);
    prof_begin("emit_partition", s);
    hipLaunchKernelGGL(k_tile_first, dim3((blocks + kBlock - 1) / kBlock), dim3(kBlock), 0, s, pair_off, n, npairs,
                       blocks, tile_first);
    prof_end("emit_partition", s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    prof_begin("emit", s);
    hipLaunchKernelGGL(k_emit, dim3(blocks), dim3(kBlock), 0, s, pair_off, box, n, npairs, tile_first, g, keys, gids,
                       pass0);
    prof_end("emit", s);
    return hipGetLastError();
}

}  // namespace gs
