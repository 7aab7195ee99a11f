// Cell index of the Gaussians (paper Sec. 4.1.1 and Sec. 4.1.2):
//  - preprocess: per Gaussian, the axis-aligned box of its cutoff ellipsoid
//    in cells (canonical float32, each operation rounded separately), its
//    cell count, and the evaluation record used by the samplers;
//  - row spans: boxes of at most kSpanRows (y, z) rows of at most kSpanNx
//    cells keep, per row, only the run of cells a float64 bound of the
//    cutoff ellipsoid's section over the row's slab can reach;
//  - emit: one (cell key, Gaussian id) pair per listed cell of every box,
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

// Minimum over the rectangle [Y0, Y1] x [Z0, Z1] of the quadratic form
// P00 y^2 + 2 P01 y z + P11 z^2 (positive definite): 0 when the origin is
// inside, else the least of the four edge minima (each a clamped 1D vertex).
__device__ double rect_qmin(double P00, double P01, double P11, double kz, double ky, double Y0, double Y1,
                            double Z0, double Z1) {
    if (Y0 <= 0.0 && 0.0 <= Y1 && Z0 <= 0.0 && 0.0 <= Z1) return 0.0;
    double best = __builtin_inf();
    const double Ys[2] = {Y0, Y1}, Zs[2] = {Z0, Z1};
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const double Y = Ys[e];
        double zs = kz * Y;
        zs = zs < Z0 ? Z0 : (zs > Z1 ? Z1 : zs);
        const double v = ((P00 * Y) * Y + 2.0 * ((P01 * Y) * zs)) + (P11 * zs) * zs;
        best = v < best ? v : best;
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const double Z = Zs[e];
        double ys = ky * Z;
        ys = ys < Y0 ? Y0 : (ys > Y1 ? Y1 : ys);
        const double v = ((P00 * ys) * ys + 2.0 * ((P01 * ys) * Z)) + (P11 * Z) * Z;
        best = v < best ? v : best;
    }
    return best;
}

// Row spans of a box (the box refined per x-row, Sec. 4.1.1). The cutoff
// ellipsoid, enlarged like the box to Q <= rci^2, meets a row's slab
// y in [y0, y1], z in [z0, z1] in a convex set. Conditioned on (y, z), x is
// centred on mu_x + b . (dy, dz) with half-width sqrt((T' - Q2) vc), Q2 the
// quadratic form of the (y, z) marginal, b = Sigma_x,yz Sigma_yz^-1 and vc
// the conditional variance; the row keeps the cells of
// [min c - wm, max c + wm], wm = sqrt((T' - min Q2) vc), with min Q2 over the
// slab's rectangle and the extremes of c at its corners, or none when
// min Q2 > T'. float64 throughout, each operation in this order. Returns
// false (box not trimmed) for boxes with more than kSpanRows rows or kSpanNx
// cells per row, or a degenerate marginal.
__device__ bool row_spans(const float mu[3], const float s[3], const float q[4], const int lo_c[3],
                          const int hi_c[3], const GridParams &g, float rci, uint8_t *__restrict__ out,
                          uint64_t &count) {
    const int nx = hi_c[0] - lo_c[0] + 1, ny = hi_c[1] - lo_c[1] + 1, nz = hi_c[2] - lo_c[2] + 1;
    if (ny * nz > kSpanRows || nx > kSpanNx) return false;
    const double qw = q[0], qx = q[1], qy = q[2], qz = q[3];
    const double qn = sqrt(((qw * qw + qx * qx) + qy * qy) + qz * qz);
    const double w = qw / qn, x = qx / qn, y = qy / qn, z = qz / qn;
    double R[3][3];
    R[0][0] = 1.0 - 2.0 * (y * y + z * z);
    R[0][1] = 2.0 * (x * y - w * z);
    R[0][2] = 2.0 * (x * z + w * y);
    R[1][0] = 2.0 * (x * y + w * z);
    R[1][1] = 1.0 - 2.0 * (x * x + z * z);
    R[1][2] = 2.0 * (y * z - w * x);
    R[2][0] = 2.0 * (x * z - w * y);
    R[2][1] = 2.0 * (y * z + w * x);
    R[2][2] = 1.0 - 2.0 * (x * x + y * y);
    double a[3][3], S[3][3];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int m = 0; m < 3; ++m) a[j][m] = R[j][m] * (double)s[m];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int k = 0; k < 3; ++k) S[j][k] = ((a[j][0] * a[k][0]) + (a[j][1] * a[k][1])) + (a[j][2] * a[k][2]);
    const double det = S[1][1] * S[2][2] - S[1][2] * S[1][2];
    if (!(det > 0.0) || !__builtin_isfinite(det)) return false;
    const double by = (S[0][1] * S[2][2] - S[0][2] * S[1][2]) / det;
    const double bz = (S[0][2] * S[1][1] - S[0][1] * S[1][2]) / det;
    const double vc = S[0][0] - (by * S[0][1] + bz * S[0][2]);
    if (!(vc > 0.0) || !__builtin_isfinite(vc)) return false;
    const double P00 = S[2][2] / det, P01 = -S[1][2] / det, P11 = S[1][1] / det;
    const double kz = -(P01 / P11), ky = -(P01 / P00);  // edge vertices: z = kz y, y = ky z
    const double Tq = (double)rci * (double)rci;
    const double icx = (double)g.cells[0] / ((double)g.hi[0] - (double)g.lo[0]);
    const double wdy = ((double)g.hi[1] - (double)g.lo[1]) / (double)g.cells[1];
    const double wdz = ((double)g.hi[2] - (double)g.lo[2]) / (double)g.cells[2];
    uint64_t cnt = 0;
    // every row byte starts empty; rows of the box are then written in turn
    const uint32_t e4 = kSpanEmpty * 0x01010101u;
#pragma unroll
    for (int k = 0; k < kSpanRows / 16; ++k) ((uint4 *)out)[k] = make_uint4(e4, e4, e4, e4);
    // rows r = (cy - y0) + ny (cz - z0), in increasing r
    int r = 0;
    for (int cz = lo_c[2]; cz <= hi_c[2]; ++cz)
    for (int cy = lo_c[1]; cy <= hi_c[1]; ++cy, ++r) {
        const double Y0 = ((double)g.lo[1] + (double)cy * wdy) - (double)mu[1];
        const double Y1 = ((double)g.lo[1] + (double)(cy + 1) * wdy) - (double)mu[1];
        const double Z0 = ((double)g.lo[2] + (double)cz * wdz) - (double)mu[2];
        const double Z1 = ((double)g.lo[2] + (double)(cz + 1) * wdz) - (double)mu[2];
        const double qmin = rect_qmin(P00, P01, P11, kz, ky, Y0, Y1, Z0, Z1);
        uint32_t code = kSpanEmpty;
        if (!(qmin > Tq)) {
            int cl = lo_c[0], ch = hi_c[0];
            const double wm = sqrt((Tq - qmin) * vc);
            const double c00 = (double)mu[0] + (by * Y0 + bz * Z0), c01 = (double)mu[0] + (by * Y0 + bz * Z1);
            const double c10 = (double)mu[0] + (by * Y1 + bz * Z0), c11 = (double)mu[0] + (by * Y1 + bz * Z1);
            const double m0 = c00 < c01 ? c00 : c01, m1 = c10 < c11 ? c10 : c11;
            const double M0 = c00 > c01 ? c00 : c01, M1 = c10 > c11 ? c10 : c11;
            const double cmin = m0 < m1 ? m0 : m1, cmax = M0 > M1 ? M0 : M1;
            const double fl = floor(((cmin - wm) - (double)g.lo[0]) * icx);
            const double fh = floor(((cmax + wm) - (double)g.lo[0]) * icx);
            if (__builtin_isfinite(fl) && __builtin_isfinite(fh)) {
                cl = fl < (double)lo_c[0] ? lo_c[0] : (fl > (double)hi_c[0] ? hi_c[0] + 1 : (int)fl);
                ch = fh > (double)hi_c[0] ? hi_c[0] : (fh < (double)lo_c[0] ? lo_c[0] - 1 : (int)fh);
            }
            if (cl <= ch) {
                code = (uint32_t)(cl - lo_c[0]) | ((uint32_t)(ch - lo_c[0]) << 4);
                cnt += (uint64_t)(ch - cl + 1);
            }
        }
        out[r] = (uint8_t)code;
    }
    count = cnt;
    return true;
}

__global__ __launch_bounds__(kBlock) void k_preprocess(const float *__restrict__ mean, const float *__restrict__ scale,
                                                       const float *__restrict__ rot, const float *__restrict__ value,
                                                       const float *__restrict__ weight, int64_t n, GridParams g,
                                                       float rci, Record *__restrict__ rec, CellBox *__restrict__ box,
                                                       uint8_t *__restrict__ spans, uint64_t *__restrict__ count) {
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
    bool trimmed = false;
    if (valid) {
        uint64_t tc = 0;
        trimmed = row_spans(mu, s, q, lo_c, hi_c, g, rci, spans + (size_t)i * kSpanRows, tc);
        if (trimmed) cnt = tc;
    }
    count[i] = cnt;
    CellBox b;
    b.lo = make_int4(lo_c[0], lo_c[1], lo_c[2], trimmed ? 1 : 0);
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

// In-place inclusive max-scan of a tile's kExpandTile marks (kExpandItems
// consecutive marks per thread, then across the block).
__device__ void tile_max_scan(uint32_t *mark, uint32_t *wmax) {
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    uint32_t run = 0;
    const uint32_t b0 = tid * kExpandItems;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t h = mark[b0 + i];
        run = h > run ? h : run;
        mark[b0 + i] = run;
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
        const uint32_t h = mark[b0 + i];
        mark[b0 + i] = h > carry ? h : carry;
    }
    __syncthreads();
}

// Row marks of trimmed boxes: at the first slot p of the tile covered by a
// non-empty row (its first pair, or slot 0 for a row begun in an earlier
// tile) the mark ((p + 1) << 16) | (row << 8) | (first << 4) | (p - start)
// holds the row, the offset of its first cell and how far into the row
// slot p is. Marks grow with p, so a max-scan hands every slot the mark of
// its row.
__device__ void mark_rows(const uint8_t *sp, uint32_t nrows, int64_t base, uint32_t tile_cnt, uint32_t *rowmark) {
    int64_t start = base;
#pragma unroll 8
    for (uint32_t r = 0; r < nrows; ++r) {
        const uint32_t code = sp[r];
        const uint32_t len = span_len(code);
        if (len > 0 && start + len > 0 && start < (int64_t)tile_cnt) {
            const uint32_t p = start > 0 ? (uint32_t)start : 0u;
            rowmark[p] = ((p + 1u) << 16) | (r << 8) | (span_first(code) << 4) | (uint32_t)((int64_t)p - start);
        }
        start += len;
    }
}

__global__ __launch_bounds__(kBlock) void k_emit(const uint64_t *__restrict__ pair_off,
                                                 const CellBox *__restrict__ box,
                                                 const uint8_t *__restrict__ spans, int64_t n, int64_t npairs,
                                                 const uint32_t *__restrict__ tile_first, GridParams g,
                                                 uint32_t *__restrict__ keys, uint32_t *__restrict__ gids,
                                                 RadixPass0 pass0) {
    __shared__ uint32_t head[kExpandTile];
    __shared__ uint32_t rowmark[kExpandTile];
    __shared__ uint32_t wmax[kWavesPerBlock];
    __shared__ uint32_t hist_lds[kMaxDigits];
    Pass0Hist hist(hist_lds, pass0);
    const uint32_t tid = threadIdx.x;
    const uint32_t tile = xcd_block(blockIdx.x, gridDim.x);
    const uint64_t tile_begin = (uint64_t)tile * kExpandTile;
    const uint64_t rem = (uint64_t)npairs - tile_begin;
    const uint32_t tile_cnt = rem < (uint64_t)kExpandTile ? (uint32_t)rem : (uint32_t)kExpandTile;
    const int64_t gfirst = tile_first[tile];
    const int64_t glast = (tile + 1 < gridDim.x) ? (int64_t)tile_first[tile + 1] : n - 1;
    for (uint32_t s = tid; s < (uint32_t)kExpandTile; s += kBlock) {
        head[s] = 0;
        rowmark[s] = 0;
    }
    __syncthreads();
    // mark the first pair of every Gaussian that starts inside the tile, and
    // the rows of the trimmed boxes that reach into it
    for (int64_t gg = gfirst + tid; gg <= glast; gg += kBlock) {
        const int64_t base = (int64_t)(pair_off[gg] - tile_begin);
        if (gg > gfirst && base < (int64_t)tile_cnt) atomicMax(&head[base], (uint32_t)(gg - gfirst));
        const CellBox b = box[gg];
        if (b.lo.w && b.hi.x >= b.lo.x) {
            const uint32_t nrows = (uint32_t)((b.hi.y - b.lo.y + 1) * (b.hi.z - b.lo.z + 1));
            mark_rows(spans + (size_t)gg * kSpanRows, nrows, base, tile_cnt, rowmark);
        }
    }
    __syncthreads();
    // inclusive max-scans carry each mark over its Gaussian's (row's) pairs
    tile_max_scan(head, wmax);
    tile_max_scan(rowmark, wmax);
    const int64_t Cx = g.cells[0], Cy = g.cells[1];
#pragma unroll 2
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t slot = (uint32_t)i * kBlock + tid;
        if (slot < tile_cnt) {
            const int64_t gg = gfirst + head[slot];
            const CellBox b = box[gg];
            const uint32_t nx = (uint32_t)(b.hi.x - b.lo.x + 1), ny = (uint32_t)(b.hi.y - b.lo.y + 1);
            uint32_t t, xo;
            if (b.lo.w) {
                const uint32_t m = rowmark[slot];
                const uint32_t p = (m >> 16) - 1u;
                t = (m >> 8) & 63u;
                xo = ((m >> 4) & 15u) + (m & 15u) + (slot - p);
            } else {
                const uint32_t local = (uint32_t)(tile_begin + slot - pair_off[gg]);
                t = local / nx;
                xo = local - t * nx;
            }
            const int64_t cx = b.lo.x + (int64_t)xo;
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
                             CellBox *box, uint8_t *spans, uint64_t *count, hipStream_t s) {
    const int64_t threads = n + 1;
    const uint32_t blocks = (uint32_t)((threads + kBlock - 1) / kBlock);
    prof_begin("preprocess", s);
    hipLaunchKernelGGL(k_preprocess, dim3(blocks), dim3(kBlock), 0, s, mean, scale, rot, value, weight, n, g, rci, rec,
                       box, spans, count);
    prof_end("preprocess", s);
    return hipGetLastError();
}

hipError_t launch_emit(const uint64_t *pair_off, const CellBox *box, const uint8_t *spans, int64_t n, int64_t npairs,
                       const GridParams &g, uint32_t *tile_first, uint32_t *keys, uint32_t *gids,
                       const RadixPass0 &pass0, hipStream_t s) {
    if (npairs <= 0 || n <= 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((npairs + kExpandTile - 1) / kExpandTile);
    prof_begin("emit_partition", s);
    hipLaunchKernelGGL(k_tile_first, dim3((blocks + kBlock - 1) / kBlock), dim3(kBlock), 0, s, pair_off, n, npairs,
                       blocks, tile_first);
    prof_end("emit_partition", s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    prof_begin("emit", s);
    hipLaunchKernelGGL(k_emit, dim3(blocks), dim3(kBlock), 0, s, pair_off, box, spans, n, npairs, tile_first, g, keys,
                       gids, pass0);
    prof_end("emit", s);
    return hipGetLastError();
}

}  // namespace gs
