// Cell index of the Gaussians (paper Sec. 4.1.1 and Sec. 4.1.2):
//  - preprocess: per Gaussian, the axis-aligned box of its cutoff ellipsoid
//    in cells (canonical float32, each operation rounded separately), its
//    cell count, and the evaluation record used by the samplers;
//  - row runs: every box of at most kTrimRowsMax (y, z) rows keeps, per
//    row, only the run of cells the cutoff ellipsoid reaches over the row's
//    slab (its exact x-extent there, in float64); the preprocess counts
//    them, the emit recomputes them;
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

// Row runs of a box (the box refined per x-row, Sec. 4.1.1). The cutoff
// ellipsoid, enlarged like the box to Q <= Tq = rci^2, meets a row's slab
// y in [Y0, Y1], z in [Z0, Z1] (offsets from the mean) in a convex set.
// Conditioned on (y, z), x is centred on by y + bz z with half-width
// sqrt((Tq - Q2) vc), Q2 the quadratic form of the (y, z) marginal and vc
// the conditional variance; the row keeps the cells of
// [min c - wm, max c + wm], wm = sqrt((Tq - min Q2) vc), with min Q2 over
// the slab's rectangle and the extremes of the centre c at its corners, or
// none when min Q2 > Tq. float64 throughout, each operation in this order.
// Boxes with a degenerate marginal, or more than kTrimRowsMax rows, keep
// every cell.
struct SpanRec {
    double P00, P01, P11;  // the (y, z) marginal's quadratic form
    double kz, ky;         // its minimisers along the rectangle's edges: z = kz y, y = ky z
    double by, bz, vc;     // x | (y, z): centre by y + bz z, variance vc
};

__device__ bool span_setup(const float s[3], const float q[4], SpanRec &p) {
    const double qw = q[0], qx = q[1], qy = q[2], qz = q[3];
    const double qn = sqrt(((qw * qw + qx * qx) + qy * qy) + qz * qz);
    const double iq = 1.0 / qn;
    const double w = qw * iq, x = qx * iq, y = qy * iq, z = qz * iq;
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
    const double idet = 1.0 / det;
    p.by = (S[0][1] * S[2][2] - S[0][2] * S[1][2]) * idet;
    p.bz = (S[0][2] * S[1][1] - S[0][1] * S[1][2]) * idet;
    p.vc = S[0][0] - (p.by * S[0][1] + p.bz * S[0][2]);
    if (!(p.vc > 0.0) || !__builtin_isfinite(p.vc)) return false;
    p.P00 = S[2][2] * idet;
    p.P01 = -S[1][2] * idet;
    p.P11 = S[1][1] * idet;
    p.kz = -(p.P01 / p.P11);
    p.ky = -(p.P01 / p.P00);
    return true;
}

// The grid in float64 for the row runs, and the enlarged cutoff.
struct SpanGrid {
    double glo[3], icx, wdy, wdz, Tq;
};

__device__ __forceinline__ SpanGrid span_grid(const GridParams &g, float rci) {
    SpanGrid sg;
    sg.glo[0] = (double)g.lo[0];
    sg.glo[1] = (double)g.lo[1];
    sg.glo[2] = (double)g.lo[2];
    sg.icx = (double)g.cells[0] / ((double)g.hi[0] - (double)g.lo[0]);
    sg.wdy = ((double)g.hi[1] - (double)g.lo[1]) / (double)g.cells[1];
    sg.wdz = ((double)g.hi[2] - (double)g.lo[2]) / (double)g.cells[2];
    sg.Tq = (double)rci * (double)rci;
    return sg;
}

// Cells of row (cy, cz) of a trimmed box spanning x0..x1 along x: their
// number, and the first as an offset from x0.
__device__ uint32_t row_cells(const SpanRec &p, const float mu[3], int x0, int x1, int cy, int cz,
                              const SpanGrid &sg, uint32_t &first) {
    first = 0;
    const double Y0 = (sg.glo[1] + (double)cy * sg.wdy) - (double)mu[1];
    const double Y1 = (sg.glo[1] + (double)(cy + 1) * sg.wdy) - (double)mu[1];
    const double Z0 = (sg.glo[2] + (double)cz * sg.wdz) - (double)mu[2];
    const double Z1 = (sg.glo[2] + (double)(cz + 1) * sg.wdz) - (double)mu[2];
    const double qmin = rect_qmin(p.P00, p.P01, p.P11, p.kz, p.ky, Y0, Y1, Z0, Z1);
    if (qmin > sg.Tq) return 0;
    const double wm = sqrt((sg.Tq - qmin) * p.vc);
    const double mx = (double)mu[0];
    const double c00 = mx + (p.by * Y0 + p.bz * Z0), c01 = mx + (p.by * Y0 + p.bz * Z1);
    const double c10 = mx + (p.by * Y1 + p.bz * Z0), c11 = mx + (p.by * Y1 + p.bz * Z1);
    const double m0 = c00 < c01 ? c00 : c01, m1 = c10 < c11 ? c10 : c11;
    const double M0 = c00 > c01 ? c00 : c01, M1 = c10 > c11 ? c10 : c11;
    const double cmin = m0 < m1 ? m0 : m1, cmax = M0 > M1 ? M0 : M1;
    const double fl = floor(((cmin - wm) - sg.glo[0]) * sg.icx), fh = floor(((cmax + wm) - sg.glo[0]) * sg.icx);
    int cl = x0, ch = x1;
    if (__builtin_isfinite(fl) && __builtin_isfinite(fh)) {
        cl = fl < (double)x0 ? x0 : (fl > (double)x1 ? x1 + 1 : (int)fl);
        ch = fh > (double)x1 ? x1 : (fh < (double)x0 ? x0 - 1 : (int)fh);
    }
    if (cl > ch) return 0;
    first = (uint32_t)(cl - x0);
    return (uint32_t)(ch - cl + 1);
}

// The rows of the wave's boxes, lane l contributing R rows (its box's, 0
// for none), walked 64 at a time in lane order. For each row, cells(o, r,
// first) gives the number of cells of row r of lane o's box (and the first
// one); visit(o, r, first, len, pos, nth) follows for every row with cells,
// pos and nth being the cells and the rows with cells among lane o's
// earlier rows (nth only when count_rows, which must be wave-uniform).
// acc and nrow are the wave's 64 LDS words each; they end holding every
// lane's totals (nrow only when count_rows).
template <class Cells, class Visit>
__device__ __forceinline__ void walk_rows(uint32_t R, uint32_t lane, uint32_t *acc, uint32_t *nrow, bool count_rows,
                                          Cells &&cells, Visit &&visit) {
    const uint32_t incl = wave_incl_sum(R);
    const uint32_t E = __builtin_amdgcn_readlane(incl, kWave - 1);
    const uint32_t excl = incl - R;
    acc[lane] = 0;
    nrow[lane] = 0;
    __builtin_amdgcn_wave_barrier();
    uint32_t j0 = 0;  // first box whose rows are not finished before the window
    for (uint32_t e0 = 0; e0 < E; e0 += kWave) {
        while (j0 + 1 < (uint32_t)kWave && __builtin_amdgcn_readlane(incl, j0) <= e0) ++j0;
        const uint32_t e = e0 + lane;
        // owner box o of element e and the element where o's rows begin
        uint32_t o = j0, base = __builtin_amdgcn_readlane(excl, j0);
        for (uint32_t jb = j0; jb + 1 < (uint32_t)kWave; ++jb) {
            const uint32_t bnd = __builtin_amdgcn_readlane(incl, jb);
            if (bnd >= e0 + kWave) break;
            if (e >= bnd) {
                o = jb + 1;
                base = bnd;
            }
        }
        const bool live = e < E;
        uint32_t first = 0, len = 0;
        if (live) len = cells(o, e - base, first);
        // the owner's earlier rows: those of past windows, then a prefix
        // over the owner's lanes of this window (from lane s0 on)
        const uint32_t has = len > 0 ? 1u : 0u;
        const uint32_t il = wave_incl_sum(len), ex = il - len;
        const uint32_t s0 = base > e0 ? base - e0 : 0u;
        const uint32_t pos = acc[o] + (ex - (uint32_t)__shfl((int)ex, (int)s0, kWave));
        uint32_t nth = 0;
        if (count_rows) {
            const uint32_t eh = wave_incl_sum(has) - has;
            nth = nrow[o] + (eh - (uint32_t)__shfl((int)eh, (int)s0, kWave));
        }
        if (live && len > 0) visit(o, e - base, first, len, pos, nth);
        const uint32_t on = (uint32_t)__shfl_down((int)o, 1u, kWave);
        const bool last = live && (lane == kWave - 1 || e + 1 == E || on != o);
        __builtin_amdgcn_wave_barrier();
        if (last) {
            acc[o] = pos + len;
            nrow[o] = nth + has;
        }
        __builtin_amdgcn_wave_barrier();
    }
}

constexpr int kPreBlock = kWave;  // one wave per workgroup: the row walk is per wave

__global__ __launch_bounds__(kPreBlock) void k_preprocess(const float *__restrict__ mean, const float *__restrict__ scale,
                                                       const float *__restrict__ rot, const float *__restrict__ value,
                                                       const float *__restrict__ weight, int64_t n, GridParams g,
                                                       float rci, Record *__restrict__ rec, CellBox *__restrict__ box,
                                                       uint8_t *__restrict__ lines, RowRec *__restrict__ rows,
                                                       uint32_t *__restrict__ rbase, uint32_t *__restrict__ rtotal,
                                                       int64_t rcap, uint8_t *__restrict__ cell_coarse,
                                                       uint64_t *__restrict__ count,
                                                       uint64_t *__restrict__ block_sum) {
    // row-run parameters and boxes of the wave's Gaussians, for the lanes
    // that walk their rows
    __shared__ SpanRec s_sp[kPreBlock];
    __shared__ float s_mu[3][kPreBlock];
    __shared__ int s_box[4][kPreBlock];  // x0, x1, y0, z0
    __shared__ uint32_t s_ny[kPreBlock];
    __shared__ uint32_t s_acc[kPreBlock], s_nrow[kPreBlock], s_rb[kPreBlock], s_trim[kPreBlock];
    // run bytes of the trim-1 boxes, word w of box t holding rows 4w..4w+3
    __shared__ uint32_t s_code[kLineRows / 4][kPreBlock];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t tid = threadIdx.x, lane = tid % kWave;
    if (i == 0) count[n] = 0;  // the element after the last count, for the offsets' scan
    const bool active = i < n;
    float mu[3] = {0.0f, 0.0f, 0.0f}, s[3] = {1.0f, 1.0f, 1.0f}, q[4] = {1.0f, 0.0f, 0.0f, 0.0f};
    float v = 0.0f, w = 0.0f;
    if (active) {
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            mu[j] = mean[3 * i + j];
            s[j] = scale[3 * i + j];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) q[j] = rot[4 * i + j];
        v = value[i];
        w = weight[i];
    }

    bool valid = active && finite_f(v) && finite_f(w);
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
    // row runs: every lane sets up its box, then the wave walks the rows of
    // all its trimmed boxes 64 at a time
    const SpanGrid sg = span_grid(g, rci);
    uint32_t nrows = 0, trim = 0;
    if (valid) {
        const int nx = hi_c[0] - lo_c[0] + 1;
        nrows = (uint32_t)((hi_c[1] - lo_c[1] + 1) * (hi_c[2] - lo_c[2] + 1));
        SpanRec sp;
        if (nrows <= kTrimRowsMax && nx <= (int)kRecNxMax && span_setup(s, q, sp)) {
            s_sp[tid] = sp;
            trim = nrows <= kLineRows && nx <= (int)kLineNx ? 1u : 2u;
        }
    }
    // trim-2 boxes: row records, one per row with cells, in a stretch of
    // as many records as the box has rows that the wave takes with one
    // atomic add (the stretches' order varies from run to run; what each
    // box finds in its own does not). A box whose stretch would pass the
    // index capacity keeps every cell instead.
    uint32_t rsum;
    {
        const uint32_t need = trim == 2 ? nrows : 0u;
        const uint32_t rincl = wave_incl_sum(need);
        rsum = __builtin_amdgcn_readlane(rincl, kWave - 1);
        uint32_t wb = 0;
        if (rsum > 0 && lane == kWave - 1) wb = atomicAdd(rtotal, rsum);
        wb = __builtin_amdgcn_readlane(wb, kWave - 1);
        const uint64_t at = (uint64_t)wb + (rincl - need);
        if (trim == 2 && at + need > (uint64_t)rcap) trim = 0;
        s_rb[tid] = (uint32_t)at;
        if (trim == 2) rbase[i] = (uint32_t)at;
    }
    if (trim == 0) nrows = 0;
    s_trim[tid] = trim;
    s_mu[0][tid] = mu[0];
    s_mu[1][tid] = mu[1];
    s_mu[2][tid] = mu[2];
    s_box[0][tid] = lo_c[0];
    s_box[1][tid] = hi_c[0];
    s_box[2][tid] = lo_c[1];
    s_box[3][tid] = lo_c[2];
    s_ny[tid] = (uint32_t)(hi_c[1] - lo_c[1] + 1);
#pragma unroll
    for (uint32_t k = 0; k < kLineRows / 4; ++k) s_code[k][tid] = kRunEmpty * 0x01010101u;
    __builtin_amdgcn_wave_barrier();
    // the cells and the rows with cells of every trimmed box; the run bytes
    // of the trim-1 boxes, the row records of the trim-2 boxes
    walk_rows(
        nrows, lane, s_acc, s_nrow, rsum > 0,
        [&](uint32_t o, uint32_t r, uint32_t &first) {
            const float mo[3] = {s_mu[0][o], s_mu[1][o], s_mu[2][o]};
            const uint32_t ny = s_ny[o], zz = r / ny;
            return row_cells(s_sp[o], mo, s_box[0][o], s_box[1][o], s_box[2][o] + (int)(r - zz * ny),
                             s_box[3][o] + (int)zz, sg, first);
        },
        [&](uint32_t o, uint32_t r, uint32_t first, uint32_t len, uint32_t pos, uint32_t nth) {
            if (s_trim[o] == 1) {
                ((uint8_t *)&s_code[r >> 2][o])[r & 3] = (uint8_t)(first | ((first + len - 1) << 4));
            } else {
                RowRec rr;
                rr.pos = pos;
                rr.row = (uint16_t)r;
                rr.first = (uint16_t)first;
                rows[(size_t)s_rb[o] + nth] = rr;
            }
        });
    __builtin_amdgcn_wave_barrier();
    uint32_t nrec = 0;
    if (trim != 0) cnt = s_acc[tid];
    if (trim == 2) nrec = s_nrow[tid];
    if (trim == 1) {
        uint4 *dst = (uint4 *)(lines + (size_t)i * kLineRows);
#pragma unroll
        for (uint32_t k = 0; k < kLineRows / 16; ++k)
            dst[k] = make_uint4(s_code[4 * k][tid], s_code[4 * k + 1][tid], s_code[4 * k + 2][tid],
                                s_code[4 * k + 3][tid]);
    }
    // the workgroup's pair count (one wave), for the offsets' scan
    {
        const uint64_t tot = wave_incl_sum64(active ? cnt : 0ull);
        if (lane == kWave - 1) block_sum[blockIdx.x] = tot;
    }
    if (!active) return;
    count[i] = cnt;
    CellBox b;
    b.lo = make_int4(lo_c[0], lo_c[1], lo_c[2], (int)trim);
    b.hi = make_int4(hi_c[0], hi_c[1], hi_c[2], (int)nrec);
    box[i] = b;

    // evaluation record: the Cholesky factor of the inverse covariance,
    // formed in float64, scaled by kRecScale and rounded once to float32
    if (valid) {
        const double qn = sqrt((double)q[0] * q[0] + (double)q[1] * q[1] + (double)q[2] * q[2] + (double)q[3] * q[3]);
        const double iq = 1.0 / qn;
        const double w_ = q[0] * iq, x = q[1] * iq, y = q[2] * iq, z = q[3] * iq;
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
        // the inverse covariance A = R S^-2 R^T and its Cholesky factor U
        // (upper triangular, A = U^T U)
        double A[3][3];
#pragma unroll
        for (int j = 0; j < 3; ++j)
#pragma unroll
            for (int l = 0; l < 3; ++l) {
                double acc = 0.0;
#pragma unroll
                for (int k = 0; k < 3; ++k) acc += Rd[j][k] * Rd[l][k] / ((double)s[k] * (double)s[k]);
                A[j][l] = acc;
            }
        const double u00 = sqrt(A[0][0]);
        const double u01 = A[0][1] / u00, u02 = A[0][2] / u00;
        const double u11 = sqrt(A[1][1] - u01 * u01);
        const double u12 = (A[1][2] - u01 * u02) / u11;
        const double u22 = sqrt(A[2][2] - u02 * u02 - u12 * u12);
        Record f;
        f.f0 = make_float4(mu[0], mu[1], mu[2], w);
        f.f1 = make_float4((float)(kRecScale * u00), (float)(kRecScale * u01), (float)(kRecScale * u02), w * v);
        f.f2 = make_float4((float)(kRecScale * u11), (float)(kRecScale * u12), (float)(kRecScale * u22), v);
        rec[i] = f;
    } else {
        Record f;
        f.f0 = f.f1 = f.f2 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        rec[i] = f;
    }
    // cells too large for the dense walk's offsets (kOffsetCells): every
    // cell of the box is marked (such a box is small against the cells;
    // concurrent marks all write 1)
    if (valid) {
        double d2 = 0.0;
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const double h = 1.0 / (double)g.invc[j];
            d2 += h * h;
        }
        const double smax = fmax(fmax((double)s[0], (double)s[1]), (double)s[2]);
        if (sqrt(d2) > kOffsetCells * smax)
            for (int z = lo_c[2]; z <= hi_c[2]; ++z)
                for (int y = lo_c[1]; y <= hi_c[1]; ++y)
                    for (int x = lo_c[0]; x <= hi_c[0]; ++x)
                        cell_coarse[(int64_t)x + g.cells[0] * ((int64_t)y + (int64_t)g.cells[1] * z)] = 1;
    }
}

// In-place inclusive max-scan of a tile's kExpandTile marks (kExpandItems
// consecutive marks per thread, then across the block).
// Inclusive max-scan of a tile of 64-bit marks in LDS (kExpandItems per
// thread, then across lanes and waves).
__device__ void tile_max_scan64(uint64_t *mark, uint64_t *wmax) {
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    uint64_t run = 0;
    const uint32_t b0 = tid * kExpandItems;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint64_t h = mark[b0 + i];
        run = h > run ? h : run;
        mark[b0 + i] = run;
    }
    uint64_t incl = run;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint64_t y = __shfl_up(incl, o, 64);
        if (lane >= (uint32_t)o) incl = y > incl ? y : incl;
    }
    uint64_t excl = __shfl_up(incl, 1, 64);
    if (lane == 0) excl = 0;
    if (lane == kWave - 1) wmax[wave] = incl;
    __syncthreads();
    uint64_t carry = excl;
    for (uint32_t w = 0; w < wave; ++w) carry = wmax[w] > carry ? wmax[w] : carry;
#pragma unroll
    for (int i = 0; i < kExpandItems; ++i) {
        const uint64_t h = mark[b0 + i];
        mark[b0 + i] = h > carry ? h : carry;
    }
    __syncthreads();
}

// Pair-parallel emit (Sec. 4.1.2): workgroup t writes pairs
// [t kExpandTile, (t + 1) kExpandTile) of the Gaussian-major list. Every row
// of cells (fixed y, z; the whole box row or its run) that reaches into the
// tile marks its first slot p in the tile with
//   (p + 1) << 52 | (Gaussian - first Gaussian of the tile) << 32 | key(p),
// so a max-scan hands every slot the mark of its row, and slot s of that row
// holds cell key(p) + s - p (keys grow by one along x). The Gaussian offset
// takes 20 bits; a tile whose Gaussian range is wider (many Gaussians without
// cells) finds the Gaussian of each slot by binary search instead.
__global__ __launch_bounds__(kBlock) void k_emit(const uint64_t *__restrict__ pair_off,
                                                 const CellBox *__restrict__ box, const uint8_t *__restrict__ lines,
                                                 const RowRec *__restrict__ rows, const uint32_t *__restrict__ rbase,
                                                 int64_t n, int64_t npairs, const uint32_t *__restrict__ tile_first,
                                                 GridParams g, uint32_t *__restrict__ keys,
                                                 uint32_t *__restrict__ gids, RadixPass0 pass0) {
    __shared__ uint64_t mark[kExpandTile];
    __shared__ uint64_t wmax[kWavesPerBlock];
    // trim-2 boxes of the current 256 Gaussians that reach into the tile:
    // their records [ja, jb) there, placed by the whole block (up to
    // kEmitTasks of them; a box past those places its records itself)
    constexpr uint32_t kEmitTasks = 64;
    __shared__ int64_t t_base[kEmitTasks];
    __shared__ uint32_t t_ja[kEmitTasks], t_jb[kEmitTasks], t_ny[kEmitTasks], t_key[kEmitTasks], t_rb[kEmitTasks];
    __shared__ uint32_t t_g[kEmitTasks];
    __shared__ uint32_t t_n;
    extern __shared__ uint32_t hist_lds[];  // the first pass's digits, sized at launch
    Pass0Hist hist(hist_lds, pass0);
    const uint32_t tid = threadIdx.x;
    const uint32_t tile = xcd_block(blockIdx.x, gridDim.x);
    const uint64_t tile_begin = (uint64_t)tile * kExpandTile;
    const uint64_t rem = (uint64_t)npairs - tile_begin;
    const uint32_t tile_cnt = rem < (uint64_t)kExpandTile ? (uint32_t)rem : (uint32_t)kExpandTile;
    const int64_t gfirst = tile_first[tile];
    const int64_t glast = (tile + 1 < gridDim.x) ? (int64_t)tile_first[tile + 1] : n - 1;
    const bool fold = glast - gfirst < ((int64_t)1 << 20);
    for (uint32_t s = tid; s < (uint32_t)kExpandTile; s += kBlock) mark[s] = 0;
    if (tid == 0) t_n = 0;
    __syncthreads();
    const int64_t Cx = g.cells[0], Cy = g.cells[1];
    const uint32_t kdz = (uint32_t)(Cx * Cy);
    for (int64_t g0 = gfirst; g0 <= glast; g0 += kBlock) {
        const int64_t gg = g0 + tid;
        // lane tid: Gaussian gg's rows of cells in the tile
        [&] {
            if (gg > glast) return;
            const int64_t base = (int64_t)(pair_off[gg] - tile_begin);  // the Gaussian's first pair, tile-relative
            const int64_t cnt = (int64_t)(pair_off[gg + 1] - pair_off[gg]);
            const CellBox b = box[gg];
            if (b.hi.x < b.lo.x || cnt == 0 || base >= (int64_t)tile_cnt || base + cnt <= 0) return;
            const uint64_t gbits = fold ? (uint64_t)(gg - gfirst) << 32 : 0ull;
            const int64_t nx = b.hi.x - b.lo.x + 1, ny = b.hi.y - b.lo.y + 1, nz = b.hi.z - b.lo.z + 1;
            // rows (y, z) are walked with counters; a row's first cell key is
            // the key of the box corner plus its offsets (keys fit 32 bits)
            const uint32_t kcorner = (uint32_t)(b.lo.x + Cx * (b.lo.y + Cy * b.lo.z));
            if (b.lo.w == 1) {
                // the runs of the box's rows, read whole from its line
                const uint4 *l4 = (const uint4 *)(lines + (size_t)gg * kLineRows);
                const uint4 c0 = l4[0], c1 = l4[1], c2 = l4[2], c3 = l4[3];
                const uint32_t words[16] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w,
                                            c2.x, c2.y, c2.z, c2.w, c3.x, c3.y, c3.z, c3.w};
                const uint32_t nrows = (uint32_t)(ny * nz);
                int64_t start = base;
                uint32_t yy = 0, krow = kcorner;  // krow: the key of the row's first box cell
                for (uint32_t r = 0; r < nrows && start < (int64_t)tile_cnt; ++r) {
                    const uint32_t code = (words[r >> 2] >> (8 * (r & 3))) & 0xFFu;
                    const uint32_t len = run_len(code);
                    if (len > 0 && start + len > 0) {
                        const int64_t p = start > 0 ? start : 0;
                        const uint32_t kp = krow + run_first(code) + (uint32_t)(p - start);
                        mark[p] = ((uint64_t)(p + 1) << 52) | gbits | (uint64_t)kp;
                    }
                    start += len;
                    if (++yy == (uint32_t)ny) {
                        yy = 0;
                        krow += kdz - (uint32_t)(Cx * (ny - 1));
                    } else {
                        krow += (uint32_t)Cx;
                    }
                }
            } else if (b.lo.w == 2) {
                // the box's records of rows with cells that reach into the tile:
                // from the last one starting at or before the tile to the last
                // one starting inside it (binary searches), as a task
                const uint32_t rb = rbase[gg];
                const RowRec *rr = rows + rb;
                const uint32_t nrec = (uint32_t)b.hi.w;
                uint32_t ja = 0;
                if (base < 0) {
                    uint32_t lo = 0, hi = nrec;  // rr[lo].pos <= -base < rr[hi].pos
                    while (hi - lo > 1) {
                        const uint32_t mid = (lo + hi) >> 1;
                        if ((int64_t)rr[mid].pos <= -base) lo = mid; else hi = mid;
                    }
                    ja = lo;
                }
                uint32_t jb = nrec;
                if (base + cnt > (int64_t)tile_cnt) {
                    uint32_t lo = ja, hi = nrec;  // rr[lo].pos < tile_cnt - base <= rr[hi].pos
                    while (hi - lo > 1) {
                        const uint32_t mid = (lo + hi) >> 1;
                        if ((int64_t)rr[mid].pos < (int64_t)tile_cnt - base) lo = mid; else hi = mid;
                    }
                    jb = hi;
                }
                const uint32_t t = atomicAdd(&t_n, 1u);
                if (t < kEmitTasks) {
                    t_base[t] = base;
                    t_ja[t] = ja;
                    t_jb[t] = jb;
                    t_ny[t] = (uint32_t)ny;
                    t_key[t] = kcorner;
                    t_rb[t] = rb;
                    t_g[t] = (uint32_t)(gg - gfirst);
                } else {
                    for (uint32_t j = ja; j < jb; ++j) {
                        const RowRec cur = rr[j];
                        const int64_t start = base + (int64_t)cur.pos;
                        const uint32_t zz = (uint32_t)cur.row / (uint32_t)ny, yy = (uint32_t)cur.row - zz * (uint32_t)ny;
                        const int64_t p = start > 0 ? start : 0;
                        const uint32_t kp =
                            kcorner + (uint32_t)Cx * yy + kdz * zz + (uint32_t)cur.first + (uint32_t)(p - start);
                        mark[p] = ((uint64_t)(p + 1) << 52) | gbits | (uint64_t)kp;
                    }
                }
            } else {
                // whole rows of nx cells: only those reaching into the tile
                const int64_t R = ny * nz;
                const int64_t r0 = base < 0 ? (-base) / nx : 0;
                int64_t r1 = ((int64_t)tile_cnt - base + nx - 1) / nx;
                r1 = r1 < R ? r1 : R;
                uint32_t yy = (uint32_t)(r0 % ny);
                uint32_t krow = kcorner + (uint32_t)Cx * yy + kdz * (uint32_t)(r0 / ny);
                for (int64_t r = r0; r < r1; ++r) {
                    const int64_t start = base + r * nx;
                    const int64_t p = start > 0 ? start : 0;
                    const uint32_t kp = krow + (uint32_t)(p - start);
                    mark[p] = ((uint64_t)(p + 1) << 52) | gbits | (uint64_t)kp;
                    if (++yy == (uint32_t)ny) {
                        yy = 0;
                        krow += kdz - (uint32_t)(Cx * (ny - 1));
                    } else {
                        krow += (uint32_t)Cx;
                    }
                }
            }

        }();
        __syncthreads();
        // the tasks' records, one per thread
        const uint32_t nt = t_n < kEmitTasks ? t_n : kEmitTasks;
        for (uint32_t t = 0; t < nt; ++t) {
            const RowRec *rr = rows + t_rb[t];
            const int64_t base = t_base[t];
            const uint32_t jb = t_jb[t], ny = t_ny[t];
            const uint64_t gbits = fold ? (uint64_t)t_g[t] << 32 : 0ull;
            for (uint32_t j = t_ja[t] + tid; j < jb; j += kBlock) {
                // every record of [ja, jb) has cells in the tile: record ja
                // ends past the tile's start, the others start inside it
                const RowRec cur = rr[j];
                const int64_t start = base + (int64_t)cur.pos;
                const uint32_t zz = (uint32_t)cur.row / ny, yy = (uint32_t)cur.row - zz * ny;
                const int64_t p = start > 0 ? start : 0;
                const uint32_t kp = t_key[t] + (uint32_t)Cx * yy + kdz * zz + (uint32_t)cur.first + (uint32_t)(p - start);
                mark[p] = ((uint64_t)(p + 1) << 52) | gbits | (uint64_t)kp;
            }
        }
        __syncthreads();
        if (tid == 0) t_n = 0;
    }
    __syncthreads();
    tile_max_scan64(mark, wmax);
#pragma unroll 2
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t slot = (uint32_t)i * kBlock + tid;
        if (slot < tile_cnt) {
            const uint64_t m = mark[slot];
            const uint32_t p = (uint32_t)(m >> 52) - 1u;
            const uint32_t key = (uint32_t)m + (slot - p);
            int64_t gg;
            if (fold)
                gg = gfirst + (int64_t)((m >> 32) & 0xFFFFFu);
            else
                gg = gfirst + segment_search(pair_off + gfirst, glast - gfirst + 1, tile_begin + slot);
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
                             const float *weight, int64_t n, const GridParams &g, float rci, Record *rec, CellBox *box,
                             uint8_t *lines, RowRec *rows, uint32_t *rbase, uint32_t *rtotal, int64_t rcap,
                             uint8_t *cell_coarse, uint64_t *count, uint64_t *block_sum, hipStream_t s) {
    // one thread per Gaussian (thread 0 also writes count[n]): for n a
    // multiple of 64 the launch fits one round of the chip
    const int64_t threads = n > 0 ? n : 1;
    const uint32_t blocks = (uint32_t)((threads + kPreBlock - 1) / kPreBlock);
    prof_begin("preprocess", s);
    hipError_t e = fill_u32(rtotal, 0u, 1, s);
    if (e == hipSuccess) e = fill_u32((uint32_t *)cell_coarse, 0u, (g.ncells + 3) / 4, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_preprocess, dim3(blocks), dim3(kPreBlock), 0, s, mean, scale, rot, value, weight, n, g, rci,
                       rec, box, lines, rows, rbase, rtotal, rcap, cell_coarse, count, block_sum);
    prof_end("preprocess", s);
    return hipGetLastError();
}

hipError_t launch_emit(const uint64_t *pair_off, const CellBox *box, const uint8_t *lines, const RowRec *rows,
                       const uint32_t *rbase, int64_t n, int64_t npairs, const GridParams &g, uint32_t *tile_first,
                       uint32_t *keys, uint32_t *gids, const RadixPass0 &pass0, hipStream_t s) {
    if (npairs <= 0 || n <= 0) return hipSuccess;
    const uint32_t blocks = (uint32_t)((npairs + kExpandTile - 1) / kExpandTile);
    prof_begin("emit", s);
    // the histogram takes only the first pass's digits: with 8-bit digits the
    // block's LDS lets 9 blocks share a compute unit instead of 7
    const size_t hist_bytes = sizeof(uint32_t) * ((size_t)pass0.mask + 1);
    hipLaunchKernelGGL(k_emit, dim3(blocks), dim3(kBlock), hist_bytes, s, pair_off, box, lines, rows, rbase, n, npairs,
                       tile_first, g, keys, gids, pass0);
    prof_end("emit", s);
    return hipGetLastError();
}

}  // namespace gs
