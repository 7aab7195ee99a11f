// Backward pass (paper Sec. 4.1.4, Fig. 4 D-E; Sec. 5.1.2).
//
// The paper assigns a thread to every (Gaussian, block) intersection, sums
// its Gaussian's partials over the block's cells and issues one atomic add
// per intersection; its unstructured backward gives each Gaussian a warp
// and ends with a warp-wide reduction. Here every Gaussian gets one
// wavefront and no atomics: the wave walks the query points in the
// Gaussian's box, accumulates the partial sums in registers and reduces
// them across the wave with DPP at the end.
//
// The queries of a Gaussian come as rows along x: for grids a row of
// voxels at fixed (y, z), contiguous in the x-fastest layout; for ordered
// queries a row of cells at fixed (y, z), contiguous in the plan's order
// (by cell, then by quarter of the cell along x). Each row is cut to the
// x-range of the cutoff ellipsoid over the row's (y, z) extent, computed
// from the Gaussian's record when the row is set up: whole voxels for
// grids, quarters of cells for ordered queries. The wave concatenates up to
// 64 rows and walks them 64 elements per step, so the lanes stay busy
// across row ends and every load reads whole cache lines. Most tested
// pairs fail the cutoff; the ones that pass are queued in LDS and
// processed 64 at a time, so the longer per-pair work runs with every lane
// busy. Gaussians are visited in the spatial order of the index (the cell
// key of their box corner), so the waves resident at one time work on one
// region and find its points in L2.
//
// Per pair the partials are kept as 11 moments in the frame of the
// record's triangular factor, u = U (p - mu) with U^T U = k^2 R S^-2 R^T
// (k^2 = log2(e) / 2), and c = dL/dQ = -1/2 a dL/da:
//   m1 = sum c u (3), m2 = sum c u u^T (6), dv = sum dL/dPhi a / I,
//   dw = sum dL/da G.
// A finalize kernel rotates them into the frame of M = S^-1 R^T (O = k M
// U^-1 is orthogonal, u / k = O^T M (p - mu)) and turns them into
// dL/dmu = -2 M^T m1,
// dL/ds_k = -2 m2_kk / s_k, dL/dR_jk = (2 / s_k) sum_m R_jm s_m m2_mk, and
// through R(qhat) and qhat = q / |q| into dL/dq.
// For a defined query with outputs (Phi, I) and cotangents (gPhi, gI):
//   dL/da_i = alpha v_i + beta with alpha = gPhi / I, beta = gI - alpha Phi,
// which a staging kernel computes once per query.
#include "internal.h"

#pragma clang fp contract(off)

namespace gs {

namespace {


__device__ __forceinline__ void alpha_beta(float phi, float inf, float gp, float gi, float &al, float &be) {
    // the forward writes I > tau > 0 at defined points and exactly 0 elsewhere
    if (inf > 0.0f) {
        al = gp / inf;
        be = gi - al * phi;
    } else {
        al = 0.0f;
        be = 0.0f;
    }
}

// Cotangents of ordered queries are first packed in query order as pairs
// (coalesced), so that staging gathers one 8-byte pair per query by id
// instead of two 4-byte values from two arrays.
constexpr int kStageItems = 4;  // queries per thread of the packing

__global__ __launch_bounds__(kBlock) void k_pack_cotangents(int64_t n, const float *__restrict__ gval,
                                                            const float *__restrict__ ginf, bool vec,
                                                            float2 *__restrict__ cot) {
    const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kStageItems;
    if (i0 >= n) return;
    if (vec && i0 + kStageItems <= n) {
        const float4 v = *(const float4 *)(gval + i0), g = *(const float4 *)(ginf + i0);
        *(float4 *)(cot + i0) = make_float4(v.x, g.x, v.y, g.y);
        *(float4 *)(cot + i0 + 2) = make_float4(v.z, g.z, v.w, g.w);
    } else {
        for (int i = 0; i < kStageItems; ++i)
            if (i0 + i < n) cot[i0 + i] = make_float2(gval[i0 + i], ginf[i0 + i]);
    }
}

// (alpha, beta) of the query at plan index k, from the forward outputs the
// plan keeps and the packed cotangents.
__global__ __launch_bounds__(kBlock) void k_stage_plan(int64_t n, const uint32_t *__restrict__ order,
                                                       const float2 *__restrict__ plan_out,
                                                       const float2 *__restrict__ cot, float2 *__restrict__ ab) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const float2 o = plan_out[k];
    // undefined queries (I = 0) have no gradient: their cotangents are not read
    const float2 c = o.y > 0.0f ? cot[order[k]] : make_float2(0.0f, 0.0f);
    float al, be;
    alpha_beta(o.x, o.y, c.x, c.y, al, be);
    ab[k] = make_float2(al, be);
}

__global__ __launch_bounds__(kBlock) void k_stage_grid(int64_t n, const float *__restrict__ value,
                                                       const float *__restrict__ influence,
                                                       const float *__restrict__ gval,
                                                       const float *__restrict__ ginf, float2 *__restrict__ ab) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float al, be;
    alpha_beta(value[i], influence[i], gval[i], ginf[i], al, be);
    ab[i] = make_float2(al, be);
}

struct Acc {
    float m1[3];
    float m2[6];  // 00 01 02 11 12 22
    float dv, dw;
};

// Whitened offset u = U (p - mu) with the record's U and Q' = |u|^2 =
// Q log2(e) / 2, Q the exponent of paper Eq. 3, as the forward forms it.
__device__ __forceinline__ float whiten(const Record &r, float px, float py, float pz, float &u0, float &u1,
                                        float &u2) {
    const float dx = px - r.f0.x, dy = py - r.f0.y, dz = pz - r.f0.z;
    u0 = fmaf_(r.f1.x, dx, fmaf_(r.f1.y, dy, r.f1.z * dz));
    u1 = fmaf_(r.f2.x, dy, r.f2.y * dz);
    u2 = r.f2.z * dz;
    return fmaf_(u0, u0, fmaf_(u1, u1, u2 * u2));
}

// Partials of one contributing pair (Q' <= T'), given u, Q' and the
// query's alpha, beta. With a = w G and dL/da = alpha v + beta, the sums
// kept are sum alpha G (dv / w), sum dL/da G (dw), and the moments of
// dL/da G u; the weight and the -1/2 of dQ/du (dL/dQ = -a dL/da / 2) are
// applied once per Gaussian by k_finalize.
__device__ __forceinline__ void pair_grad(const Record &r, float u0, float u1, float u2, float Q, float al, float be,
                                          Acc &acc) {
    const float G = exp2_hw(-Q);  // Q is Q' = Q log2(e) / 2
    const float dLda = fmaf_(al, r.f2.w, be);
    const float c = dLda * G;
    acc.dv = fmaf_(al, G, acc.dv);
    acc.dw += c;
    const float c0 = c * u0, c1 = c * u1, c2 = c * u2;
    acc.m1[0] += c0;
    acc.m1[1] += c1;
    acc.m1[2] += c2;
    acc.m2[0] = fmaf_(c0, u0, acc.m2[0]);
    acc.m2[1] = fmaf_(c0, u1, acc.m2[1]);
    acc.m2[2] = fmaf_(c0, u2, acc.m2[2]);
    acc.m2[3] = fmaf_(c1, u1, acc.m2[3]);
    acc.m2[4] = fmaf_(c1, u2, acc.m2[4]);
    acc.m2[5] = fmaf_(c2, u2, acc.m2[5]);
}

// One step of a transposed reduction: the lane keeps one of (lo, hi) by its
// lane bit and adds the partner's copy of the same element; the partner
// (reached with DPP control CTRL) differs from the lane in that bit.
template <int CTRL>
__device__ __forceinline__ float tr_step(float lo, float hi, bool bit) {
    const float keep = bit ? hi : lo, send = bit ? lo : hi;
    return keep + dpp_f<CTRL>(send);
}

// Sum of 11 per-lane values over the wave; lane k < 11 returns total k
// (lanes 11..15 return 0). Four transposed steps inside each row of 16
// (lane bits 0, 1, 2, 3 through quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_ror:4, row_ror:8) leave lane l holding element l & 15 summed over its
// row; an xor-16 swizzle and an xor-32 permute then add the four rows.
__device__ __forceinline__ float reduce11(const float v[11], uint32_t lane) {
    const bool b0 = lane & 1u, b1 = lane & 2u, b2 = lane & 4u, b3 = lane & 8u;
    float w[6];
#pragma unroll
    for (int i = 0; i < 5; ++i) w[i] = tr_step<0xB1>(v[2 * i], v[2 * i + 1], b0);
    w[5] = tr_step<0xB1>(v[10], 0.0f, b0);
    float x[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) x[j] = tr_step<0x4E>(w[2 * j], w[2 * j + 1], b1);
    const float y0 = tr_step<0x124>(x[0], x[1], b2);
    const float y1 = tr_step<0x124>(x[2], 0.0f, b2);
    float z = tr_step<0x128>(y0, y1, b3);
    z += swz_xor16(z);
    z += perm_xor32(z, lane);
    return z;
}

// Queue of contributing pairs of one wave: (u0, u1, u2, Q) and the point.
// (Loading each lane's (alpha, beta) with its position, so that the queue
// holds them instead of the point, was slower: 8 more bytes a test.)
constexpr uint32_t kQueue = 2 * kWave;

__device__ __forceinline__ void drain(const Record &r, const float4 *qu, const uint32_t *qk, uint32_t head,
                                      uint32_t cnt, uint32_t lane, const float2 *__restrict__ ab, Acc &acc) {
    if (lane < cnt) {
        const uint32_t slot = (head + lane) & (kQueue - 1);
        const float4 e = qu[slot];
        const float2 c = ab[qk[slot]];
        pair_grad(r, e.x, e.y, e.z, e.w, c.x, c.y, acc);
    }
}

// The per-Gaussian kernel runs one wave per workgroup: its waves are
// independent (each has its own LDS queue) and their costs vary with the
// Gaussians' boxes; a workgroup keeps its LDS until its slowest wave ends.
// Waves are taken in launch order (dealt round-robin over the XCDs by the
// dispatcher, four consecutive waves to an XCD), so every XCD works on the
// same stretch of the spatial order at a time rather than on a fixed eighth
// of it.
constexpr int kBwdWaves = 1;
constexpr int kBwdBlock = kBwdWaves * kWave;
// Four consecutive waves per XCD (xcd_group): neighbouring Gaussians read
// the same queries through one L2 (C4's backward about 1 % faster).
constexpr uint32_t kXcdWaves = 4;
// Element windows per step of the walk (see the window loop).
constexpr uint32_t kBwdWindows = 2;
static_assert(kBwdWindows == 2, "the walk's uniform steps take two windows");
// Mean row length (elements per row of a Gaussian's part of a batch) from
// which the walk tracks its row in scalars.
constexpr uint32_t kLongRow = 128;

// Gaussians per wavefront: consecutive Gaussians of gorder share a wave, so
// that their rows are found together. Below kPackMinGauss Gaussians one per
// wave (more would leave SIMDs idle); otherwise kPack, or kPackLarge (one)
// when the boxes list at least kLargeBoxCells cells on average (a wave's
// cost grows with its Gaussians' boxes, and one per wave balances best).
constexpr uint32_t kPack = 4;
constexpr uint32_t kPackLarge = 1;
constexpr int64_t kPackMinGauss = 65536;
constexpr int64_t kLargeBoxCells = 32;

// Partials of the wave's current Gaussian are reduced over the wave and
// stored: lane k < 12 writes moment k (the 12th is 0).
__device__ __forceinline__ void finish_gauss(const Record &r, const float4 *qu, const uint32_t *qk, uint32_t head,
                                             uint32_t cnt, uint32_t lane, const float2 *__restrict__ ab, Acc &acc,
                                             uint32_t gid, float *__restrict__ moments) {
    if (cnt > 0) {
        __builtin_amdgcn_wave_barrier();
        drain(r, qu, qk, head, cnt, lane, ab, acc);
    }
    const float v[11] = {acc.m1[0], acc.m1[1], acc.m1[2], acc.m2[0], acc.m2[1], acc.m2[2],
                         acc.m2[3], acc.m2[4], acc.m2[5], acc.dv,    acc.dw};
    const float tot = reduce11(v, lane);
    if (lane < 12) moments[(size_t)gid * 12 + lane] = tot;
}

__device__ __forceinline__ void acc_zero(Acc &acc) {
#pragma unroll
    for (int k = 0; k < 3; ++k) acc.m1[k] = 0.0f;
#pragma unroll
    for (int k = 0; k < 6; ++k) acc.m2[k] = 0.0f;
    acc.dv = acc.dw = 0.0f;
}

__device__ __forceinline__ float bperm_f(uint32_t src, float v) {
    return __int_as_float(__builtin_amdgcn_ds_bpermute((int)src, __float_as_int(v)));
}

// Row `row` of a Gaussian's box (lower corner (lx, ly, lz) in cells, nx
// cells along x, ny along y): for grids voxel row (vy, vz) of the box, for
// ordered queries the row of cells (cy, cz), y fastest. The row's first
// element (voxel index, or place in the plan's order), its length, and for
// grids its first voxel along x and the row's y, z.
struct RowRun {
    uint32_t start, len, x0;
    float py, pz;
};

template <bool GRID>
__device__ __forceinline__ RowRun row_run(const Record &r, int32_t lx, int32_t ly, int32_t lz, uint32_t nx,
                                          uint32_t ny, uint32_t row, uint32_t rx, uint32_t ry, uint32_t rz, bool fdiv,
                                          const QueryParams &q, const GridParams &g, const BwdGeom &bg,
                                          const uint32_t *__restrict__ point_off) {
    RowRun o;
    o.start = o.len = o.x0 = 0;
    o.py = o.pz = 0.0f;
    const uint32_t nry = GRID ? ny * ry : ny;
    // row -> (yy, zz) by a float reciprocal: (row + 1/2) / nry lies at least
    // 1/(2 nry) from an integer; v_rcp (1 ulp) and the product err by less
    // than 1.5 2^-23 (row + 1/2) / nry, which cannot cross it while
    // row < 2^21
    uint32_t zz;
    if (fdiv)
        zz = (uint32_t)(((float)row + 0.5f) * __builtin_amdgcn_rcpf((float)nry));
    else
        zz = row / nry;
    const uint32_t yy = row - zz * nry;
    if (GRID) {
        float xl, xh;
        (void)rz;
        const uint32_t vy = (uint32_t)ly * ry + yy, vz = (uint32_t)lz * rz + zz;
        o.py = g.lo[1] + ((float)vy + 0.5f) * q.vsz[1];
        o.pz = g.lo[2] + ((float)vz + 0.5f) * q.vsz[2];
        const float dy = o.py - r.f0.y, dz = o.pz - r.f0.z;
        if (!slab_xrange(r, dy, dy, dz, dz, bg.T2, xl, xh)) return o;
        // voxels vx of the box with lo + (vx + 1/2) vsz in [xl, xh]
        const float vmin = (float)((uint32_t)lx * rx), vmax = (float)(((uint32_t)lx + nx) * rx) - 1.0f;
        const float a = fminf(fmaxf((xl - g.lo[0]) * bg.ivsz0 - 0.5f - bg.xslack, vmin), vmax + 1.0f);
        const float b = fminf(fmaxf((xh - g.lo[0]) * bg.ivsz0 - 0.5f + bg.xslack, vmin - 1.0f), vmax);
        const float v0 = ceilf(a), v1 = floorf(b);
        if (v1 < v0) return o;
        o.x0 = (uint32_t)v0;
        o.len = (uint32_t)(v1 - v0) + 1u;
        o.start = (uint32_t)q.dims[0] * (vy + (uint32_t)q.dims[1] * vz) + o.x0;
    } else {
        o.len = plan_row(r, (uint32_t)lx, nx, (uint32_t)ly + yy, (uint32_t)lz + zz, g, bg, point_off, o.start);
    }
    return o;
}

// PACK consecutive Gaussians of gorder per wavefront. The rows of the
// wave's Gaussians are listed one Gaussian after the other and taken 64 at
// a time, lane l setting up row l of the batch (its x-range from the
// Gaussian's record, for ordered queries two offsets of the plan). Within a batch the rows are concatenated; each Gaussian walks
// its own part 64 elements per step, lane l taking element e0 + l, so the
// lanes stay busy across row ends and every load reads whole cache lines;
// a lane finds its row from the row starts with two ballots. The cutoff
// test is all a non-contributing pair costs; contributing pairs go to a
// per-wave LDS queue, and every 64 queued pairs are processed with all
// lanes busy.
template <bool GRID, uint32_t PACK>
__global__ __launch_bounds__(kBwdBlock) void k_backward_gauss(QueryParams q, GridParams g, BwdGeom bg,
                                                           const Record *__restrict__ rec,
                                                           const CellBox *__restrict__ box,
                                                           const uint32_t *__restrict__ gorder, int64_t n_gauss,
                                                           const uint32_t *__restrict__ point_off,
                                                           const float4 *__restrict__ plan_pos,
                                                           const float2 *__restrict__ ab, float T,
                                                           float *__restrict__ moments) {
    __shared__ float4 s_qu[kBwdWaves][kQueue];
    __shared__ uint32_t s_qk[kBwdWaves][kQueue];
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t wib = threadIdx.x / kWave;
    const uint64_t w = (uint64_t)xcd_group<kXcdWaves>(blockIdx.x, gridDim.x) * kBwdWaves + wib;
    const uint64_t first = w * PACK;
    if (first >= (uint64_t)n_gauss) return;
    const uint32_t nk = (uint64_t)n_gauss - first < PACK ? (uint32_t)((uint64_t)n_gauss - first) : PACK;
    float4 *qu = s_qu[wib];
    uint32_t *qk = s_qk[wib];
    uint32_t rx = 1, ry = 1, rz = 1;
    if (GRID) {
        rx = (uint32_t)(q.dims[0] / g.cells[0]);
        ry = (uint32_t)(q.dims[1] / g.cells[1]);
        rz = (uint32_t)(q.dims[2] / g.cells[2]);
    }
    // lane i < nk describes Gaussian i of the wave: id, box, rows
    uint32_t mgid = 0, mR = 0, mnx = 0, mny = 1;
    int32_t mlx = 0, mly = 0, mlz = 0;
    Record mrec;
    mrec.f0 = mrec.f1 = mrec.f2 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (lane < nk) {
        mgid = gorder[first + lane];
        mrec = rec[mgid];
        const CellBox bx = box[mgid];
        if (bx.hi.x >= bx.lo.x) {
            mnx = (uint32_t)(bx.hi.x - bx.lo.x + 1);
            mny = (uint32_t)(bx.hi.y - bx.lo.y + 1);
            const uint32_t nz = (uint32_t)(bx.hi.z - bx.lo.z + 1);
            mR = GRID ? mny * ry * nz * rz : mny * nz;
            mlx = bx.lo.x;
            mly = bx.lo.y;
            mlz = bx.lo.z;
        }
        // a Gaussian without rows gets zero moments here
        if (mR == 0) {
            float4 *m4 = (float4 *)(moments + (size_t)mgid * 12);
            const float4 z = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            m4[0] = z;
            m4[1] = z;
            m4[2] = z;
        }
    }
    const uint32_t mRend = wave_incl_sum(mR);  // end of Gaussian i's rows in the wave's list
    const uint32_t Rw = __builtin_amdgcn_readlane(mRend, kWave - 1);
    // rows -> (yy, zz) by a float reciprocal below 2^21 rows (see row_run)
    const bool fdiv = wave_max_uniform(mR) < (1u << 21);
    Record r;
    r.f0 = r.f1 = r.f2 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    Acc acc;
    acc_zero(acc);
    uint32_t head = 0, cnt = 0;
    uint32_t cur = PACK, cur_gid = 0;  // the Gaussian being walked (none yet)
    for (uint32_t rb = 0; rb < Rw; rb += kWave) {
        // lane l describes row rb + l of the wave's list: its Gaussian i is
        // the number of Gaussians whose rows end at or before it
        const uint32_t gr = rb + lane;
        uint32_t i = 0;
        for (uint32_t t = 0; t < nk; ++t) i += __builtin_amdgcn_readlane(mRend, t) <= gr ? 1u : 0u;
        const uint32_t src = (i < kWave ? i : 0u) << 2;
        const uint32_t f_end = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)mRend);
        const uint32_t f_R = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)mR);
        const uint32_t f_nx = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)mnx);
        const uint32_t f_ny = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, (int)mny);
        const uint32_t f_lx = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, mlx);
        const uint32_t f_ly = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, mly);
        const uint32_t f_lz = (uint32_t)__builtin_amdgcn_ds_bpermute((int)src, mlz);
        uint32_t start = 0, len = 0, rx0 = 0;
        float rpy = 0.0f, rpz = 0.0f;
        if (gr < Rw) {
            const uint32_t row = gr - (f_end - f_R);  // row within its Gaussian
            Record fr;
            fr.f0 = make_float4(bperm_f(src, mrec.f0.x), bperm_f(src, mrec.f0.y), bperm_f(src, mrec.f0.z), 0.0f);
            fr.f1 = make_float4(bperm_f(src, mrec.f1.x), bperm_f(src, mrec.f1.y), bperm_f(src, mrec.f1.z), 0.0f);
            fr.f2 = make_float4(bperm_f(src, mrec.f2.x), bperm_f(src, mrec.f2.y), bperm_f(src, mrec.f2.z), 0.0f);
            const RowRun rr = row_run<GRID>(fr, (int32_t)f_lx, (int32_t)f_ly, (int32_t)f_lz, f_nx, f_ny, row, rx, ry,
                                            rz, fdiv, q, g, bg, point_off);
            start = rr.start;
            len = rr.len;
            rx0 = rr.x0;
            rpy = rr.py;
            rpz = rr.pz;
        }
        const uint32_t nrows = (Rw - rb) < (uint32_t)kWave ? (Rw - rb) : (uint32_t)kWave;
        const uint32_t incl = wave_incl_sum(len);   // end of row l in the batch's concatenation
        const uint32_t E = __builtin_amdgcn_readlane(incl, kWave - 1);
        const uint32_t rbeg = incl - len;           // first element of row l
        const uint32_t kofs = start - rbeg;         // element e of row l is point e + kofs
        const uint32_t xofs = rx0 - rbeg;           // grids: element e of row l has x = e + xofs
        // the Gaussians with rows in this batch, in order
        const uint32_t ia = __builtin_amdgcn_readlane(i, 0), ib = __builtin_amdgcn_readlane(i, nrows - 1);
        for (uint32_t gi = ia; gi <= ib; ++gi) {
            const uint32_t gend = __builtin_amdgcn_readlane(mRend, gi), gR = __builtin_amdgcn_readlane(mR, gi);
            if (gR == 0) continue;  // no rows: its moments are written above
            if (gi != cur) {
                if (cur < PACK) finish_gauss(r, qu, qk, head, cnt, lane, ab, acc, cur_gid, moments);
                head = cnt = 0;
                acc_zero(acc);
                cur = gi;
                cur_gid = __builtin_amdgcn_readlane(mgid, gi);
                r = load_record_uniform(rec, cur_gid);
            }
            // its rows in this batch and their elements [Ea, Eb)
            const uint32_t la = gend - gR > rb ? gend - gR - rb : 0u;
            const uint32_t lb = gend - rb < nrows ? gend - rb : nrows;
            const uint32_t Ea = __builtin_amdgcn_readlane(rbeg, la);
            const uint32_t Eb = lb < (uint32_t)kWave ? __builtin_amdgcn_readlane(rbeg, lb) : E;
            // The element window [e0, e0 + 64): the offset of each lane's row
            // (ko: element e of the row is point e + ko; grids: x offset xo and
            // the row's y, z).
            auto locate = [&](uint32_t e0, uint32_t &ko, uint32_t &xo, float &py, float &pz) {
                // rbeg rises with the lane (lanes past nrows hold E), so the
                // rows starting at or before e0 are a prefix of the lanes and
                // the last of them holds element e0
                const uint32_t j0 = (uint32_t)__popcll(mask_le_u(rbeg, e0)) - 1u;
                const uint32_t e = e0 + lane;
                ko = __builtin_amdgcn_readlane(kofs, j0);  // row of element e0
                xo = 0;
                py = pz = 0.0f;
                if (GRID) {
                    xo = __builtin_amdgcn_readlane(xofs, j0);
                    py = readlane_f(rpy, j0);
                    pz = readlane_f(rpz, j0);
                }
                // rows starting inside the window move the later lanes on, in
                // row order (an empty row is overridden by the next)
                uint64_t inw = mask_lt_u(lane, nrows) & mask_lt_u(rbeg - e0 - 1u, (uint32_t)kWave - 1u);
                while (inw != 0) {
                    const uint32_t j = (uint32_t)__builtin_ctzll(inw);
                    inw &= inw - 1;
                    const bool nxt = e >= __builtin_amdgcn_readlane(rbeg, j);
                    ko = nxt ? __builtin_amdgcn_readlane(kofs, j) : ko;
                    if (GRID) {
                        xo = nxt ? __builtin_amdgcn_readlane(xofs, j) : xo;
                        py = nxt ? readlane_f(rpy, j) : py;
                        pz = nxt ? readlane_f(rpz, j) : pz;
                    }
                }
            };
            // The cutoff test of the window's pairs; contributing ones go to
            // the queue, which is processed 64 pairs at a time.
            auto test = [&](uint32_t e0, uint32_t ko, uint32_t xo, float py, float pz, float4 p) {
                // lanes past the Gaussian's last element read the elements
                // after it: points of later rows, or past the batch's last
                // row, whose last point is at most n - 1, up to 63 entries of
                // the plan's spare tail; their test has no effect
                const uint32_t e = e0 + lane;
                const bool valid = e < Eb;
                const uint32_t k = e + ko;
                float u0, u1, u2, Q;
                if (GRID) {
                    const float px = g.lo[0] + ((float)(e + xo) + 0.5f) * q.vsz[0];
                    Q = whiten(r, px, py, pz, u0, u1, u2);
                } else {
                    Q = whiten(r, p.x, p.y, p.z, u0, u1, u2);
                }
                const bool hit = valid && Q <= T;
                const uint64_t mask = mask_le_f(Q, T) & mask_lt_u(e, Eb);
                if (mask == 0) return;
                if (hit) {
                    const uint32_t pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                    const uint32_t slot = (head + cnt + pos) & (kQueue - 1);
                    qu[slot] = make_float4(u0, u1, u2, Q);
                    qk[slot] = k;
                }
                cnt += (uint32_t)__popcll(mask);
                if (cnt >= (uint32_t)kWave) {
                    __builtin_amdgcn_wave_barrier();
                    drain(r, qu, qk, head, kWave, lane, ab, acc);
                    __builtin_amdgcn_wave_barrier();
                    head = (head + kWave) & (kQueue - 1);
                    cnt -= kWave;
                }
            };
            // The row holding element e, tracked in scalars: its offset kos
            // and the start nxt of the row after it (lanes past the batch's
            // rows hold E).
            uint32_t kos = 0, nxt = 0;
            auto row_at = [&](uint32_t e) {
                const uint32_t j = (uint32_t)__popcll(mask_le_u(rbeg, e)) - 1u;
                kos = __builtin_amdgcn_readlane(kofs, j);
                nxt = j + 1u < (uint32_t)kWave ? __builtin_amdgcn_readlane(rbeg, j + 1u) : E;
            };
            // The test of a window that lies inside one row and before Eb:
            // every lane is valid and element e0 + l is point e0 + kos + l.
            auto test_row = [&](uint32_t e0, float4 p) {
                float u0, u1, u2;
                const float Q = whiten(r, p.x, p.y, p.z, u0, u1, u2);
                const uint64_t mask = mask_le_f(Q, T);
                if (mask == 0) return;
                if (Q <= T) {
                    const uint32_t pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                    const uint32_t slot = (head + cnt + pos) & (kQueue - 1);
                    qu[slot] = make_float4(u0, u1, u2, Q);
                    qk[slot] = e0 + kos + lane;
                }
                cnt += (uint32_t)__popcll(mask);
                if (cnt >= (uint32_t)kWave) {
                    __builtin_amdgcn_wave_barrier();
                    drain(r, qu, qk, head, kWave, lane, ab, acc);
                    __builtin_amdgcn_wave_barrier();
                    head = (head + kWave) & (kQueue - 1);
                    cnt -= kWave;
                }
            };
            // Windows are taken two at a time: both positions are loaded
            // before either is tested, so one load's latency overlaps the
            // other window's work. When the Gaussian's rows are long, a step
            // whose windows are full and inside one row (most of them then)
            // skips the per-lane row search and loads from a uniform base;
            // with short rows the scalar bookkeeping would cost more than it
            // saves.
            const bool long_rows = !GRID && Eb - Ea >= kLongRow * (lb - la);
            for (uint32_t e0 = Ea; e0 < Eb; e0 += kBwdWindows * kWave) {
                if (long_rows) {
                    if (e0 >= nxt) row_at(e0);
                    const uint32_t eend = e0 + kBwdWindows * kWave;
                    if (eend <= nxt && eend <= Eb) {
                        const float4 *pp = plan_pos + (e0 + kos);
                        const float4 pA = pp[lane], pB = pp[kWave + lane];
                        test_row(e0, pA);
                        test_row(e0 + kWave, pB);
                        continue;
                    }
                }
                uint32_t koA, xoA, koB = 0, xoB = 0;
                float pyA, pzA, pyB = 0.0f, pzB = 0.0f;
                const uint32_t e1 = e0 + kWave;
                const bool two = kBwdWindows > 1 && e1 < Eb;
                float4 pA = make_float4(0.0f, 0.0f, 0.0f, 0.0f), pB = pA;
                locate(e0, koA, xoA, pyA, pzA);
                if (!GRID) pA = plan_pos[e0 + lane + koA];
                if (two) {
                    locate(e1, koB, xoB, pyB, pzB);
                    if (!GRID) pB = plan_pos[e1 + lane + koB];
                }
                test(e0, koA, xoA, pyA, pzA, pA);
                if (two) test(e1, koB, xoB, pyB, pzB, pB);
            }
        }
    }
    if (cur < PACK) finish_gauss(r, qu, qk, head, cnt, lane, ab, acc, cur_gid, moments);
}

__global__ __launch_bounds__(kBlock) void k_finalize(const float *__restrict__ moments, int64_t n,
                                                     const Record *__restrict__ rec,
                                                     const float *__restrict__ scale, const float *__restrict__ rot,
                                                     float *__restrict__ d_mean, float *__restrict__ d_scale,
                                                     float *__restrict__ d_rot, float *__restrict__ d_value,
                                                     float *__restrict__ d_weight) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *m = moments + (size_t)i * 12;
    const float4 ma = *(const float4 *)m, mb = *(const float4 *)(m + 4), mc = *(const float4 *)(m + 8);
    // moments of dL/dQ u / k (the unscaled factor's frame): the kernel's
    // sums of dL/da G u times -w/2, over k
    constexpr double ik = 1.0 / kRecScale, ik2 = ik * ik;
    const double wt = rec[i].f0.w, c1 = -0.5 * wt * ik, c2 = -0.5 * wt * ik2;
    const double m1p[3] = {ma.x * c1, ma.y * c1, ma.z * c1};
    const double m2s[6] = {ma.w * c2, mb.x * c2, mb.y * c2, mb.z * c2, mb.w * c2, mc.x * c2};
    const bool any = ma.x != 0.0f || ma.y != 0.0f || ma.z != 0.0f || ma.w != 0.0f || mb.x != 0.0f ||
                     mb.y != 0.0f || mb.z != 0.0f || mb.w != 0.0f || mc.x != 0.0f || mc.y != 0.0f || mc.z != 0.0f;
    // the parameters are loaded with the moments, whatever these hold
    const double s[3] = {scale[3 * i], scale[3 * i + 1], scale[3 * i + 2]};
    const double q[4] = {rot[4 * i], rot[4 * i + 1], rot[4 * i + 2], rot[4 * i + 3]};
    double dmu[3] = {0, 0, 0}, ds[3] = {0, 0, 0}, dq[4] = {0, 0, 0, 0};
    if (any) {
        const double is[3] = {1.0 / s[0], 1.0 / s[1], 1.0 / s[2]};
        const double qn = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
        const double iqn = 1.0 / qn;
        const double w = q[0] * iqn, x = q[1] * iqn, y = q[2] * iqn, z = q[3] * iqn;
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
        // Scaled back by 1/k above, the moments are in the frame of u' = U d
        // for U upper triangular with U^T U = M^T M, M = S^-1 R^T (the
        // record's factor over k). O = M U^-1 is orthogonal and u = M d =
        // O u', so the moments in the frame of M are m1 = O m1' and
        // m2 = O m2' O^T.
        double Mm[3][3], A[3][3];
        for (int k = 0; k < 3; ++k)
            for (int j = 0; j < 3; ++j) Mm[k][j] = R[j][k] * is[k];
        for (int j = 0; j < 3; ++j)
            for (int l = 0; l < 3; ++l) A[j][l] = Mm[0][j] * Mm[0][l] + Mm[1][j] * Mm[1][l] + Mm[2][j] * Mm[2][l];
        const double u00 = sqrt(A[0][0]);
        const double u01 = A[0][1] / u00, u02 = A[0][2] / u00;
        const double u11 = sqrt(A[1][1] - u01 * u01);
        const double u12 = (A[1][2] - u01 * u02) / u11;
        const double u22 = sqrt(A[2][2] - u02 * u02 - u12 * u12);
        const double Ui[3][3] = {{1.0 / u00, -u01 / (u00 * u11), (u01 * u12 - u02 * u11) / (u00 * u11 * u22)},
                                 {0.0, 1.0 / u11, -u12 / (u11 * u22)},
                                 {0.0, 0.0, 1.0 / u22}};
        double O[3][3];
        for (int k = 0; k < 3; ++k)
            for (int a = 0; a < 3; ++a) O[k][a] = Mm[k][0] * Ui[0][a] + Mm[k][1] * Ui[1][a] + Mm[k][2] * Ui[2][a];
        double P2[3][3];
        P2[0][0] = m2s[0];
        P2[0][1] = P2[1][0] = m2s[1];
        P2[0][2] = P2[2][0] = m2s[2];
        P2[1][1] = m2s[3];
        P2[1][2] = P2[2][1] = m2s[4];
        P2[2][2] = m2s[5];
        double m1[3], OP[3][3], M2[3][3];
        for (int k = 0; k < 3; ++k) m1[k] = O[k][0] * m1p[0] + O[k][1] * m1p[1] + O[k][2] * m1p[2];
        for (int k = 0; k < 3; ++k)
            for (int b = 0; b < 3; ++b) OP[k][b] = O[k][0] * P2[0][b] + O[k][1] * P2[1][b] + O[k][2] * P2[2][b];
        for (int k = 0; k < 3; ++k)
            for (int l = 0; l < 3; ++l) M2[k][l] = OP[k][0] * O[l][0] + OP[k][1] * O[l][1] + OP[k][2] * O[l][2];
        for (int j = 0; j < 3; ++j) {
            double acc = 0.0;
            for (int k = 0; k < 3; ++k) acc += R[j][k] * m1[k] * is[k];
            dmu[j] = -2.0 * acc;
        }
        for (int k = 0; k < 3; ++k) ds[k] = -2.0 * M2[k][k] * is[k];
        double G[3][3];
        for (int j = 0; j < 3; ++j)
            for (int k = 0; k < 3; ++k) {
                double acc = 0.0;
                for (int mm = 0; mm < 3; ++mm) acc += R[j][mm] * s[mm] * M2[mm][k];
                G[j][k] = 2.0 * acc * is[k];
            }
        double dqh[4];
        dqh[0] = 2.0 * (-z * G[0][1] + y * G[0][2] + z * G[1][0] - x * G[1][2] - y * G[2][0] + x * G[2][1]);
        dqh[1] = 2.0 * (y * G[0][1] + z * G[0][2] + y * G[1][0] - 2.0 * x * G[1][1] - w * G[1][2] + z * G[2][0] +
                        w * G[2][1] - 2.0 * x * G[2][2]);
        dqh[2] = 2.0 * (-2.0 * y * G[0][0] + x * G[0][1] + w * G[0][2] + x * G[1][0] + z * G[1][2] - w * G[2][0] +
                        z * G[2][1] - 2.0 * y * G[2][2]);
        dqh[3] = 2.0 * (-2.0 * z * G[0][0] - w * G[0][1] + x * G[0][2] + w * G[1][0] - 2.0 * z * G[1][1] +
                        y * G[1][2] + x * G[2][0] + y * G[2][1]);
        const double dot = w * dqh[0] + x * dqh[1] + y * dqh[2] + z * dqh[3];
        const double qh[4] = {w, x, y, z};
        for (int k = 0; k < 4; ++k) dq[k] = (dqh[k] - qh[k] * dot) * iqn;
    }
    for (int j = 0; j < 3; ++j) {
        d_mean[3 * i + j] = (float)dmu[j];
        d_scale[3 * i + j] = (float)ds[j];
    }
    for (int k = 0; k < 4; ++k) d_rot[4 * i + k] = (float)dq[k];
    d_value[i] = (float)(mc.y * wt);
    d_weight[i] = mc.z;
}

// Pairs the backward tests, for measurement: per Gaussian the elements of
// its rows, each cut to its x-range as the backward cuts it (row_run).
// Summed per block, then into *total with one integer atomic per block (the
// sum does not depend on its order).
template <bool GRID>
__global__ __launch_bounds__(kBlock) void k_count_backward_pairs(QueryParams q, GridParams g, BwdGeom bg,
                                                                 const Record *__restrict__ rec,
                                                                 const CellBox *__restrict__ box, int64_t n_gauss,
                                                                 const uint32_t *__restrict__ point_off,
                                                                 unsigned long long *total) {
    __shared__ unsigned long long lds[kWavesPerBlock];
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    unsigned long long c = 0;
    if (i < n_gauss) {
        const CellBox bx = box[i];
        if (bx.hi.x >= bx.lo.x) {
            const uint32_t rx = GRID ? (uint32_t)(q.dims[0] / g.cells[0]) : 1u;
            const uint32_t ry = GRID ? (uint32_t)(q.dims[1] / g.cells[1]) : 1u;
            const uint32_t rz = GRID ? (uint32_t)(q.dims[2] / g.cells[2]) : 1u;
            const uint32_t nx = (uint32_t)(bx.hi.x - bx.lo.x + 1), ny = (uint32_t)(bx.hi.y - bx.lo.y + 1);
            const uint32_t nz = (uint32_t)(bx.hi.z - bx.lo.z + 1);
            const uint32_t R = GRID ? ny * ry * nz * rz : ny * nz;
            const Record r = rec[i];
            for (uint32_t row = 0; row < R; ++row)
                c += row_run<GRID>(r, bx.lo.x, bx.lo.y, bx.lo.z, nx, ny, row, rx, ry, rz, false, q, g, bg, point_off)
                         .len;
        }
    }
    // block sum in a fixed order, then one atomic per block
    const uint32_t lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) c += __shfl_xor(c, o, kWave);
    if (lane == 0) lds[wid] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
        for (int w = 0; w < kWavesPerBlock; ++w) t += lds[w];
        if (t) atomicAdd(total, t);
    }
}

template <bool GRID>
void launch_gauss(uint32_t pack, uint32_t wblocks, hipStream_t s, const QueryParams &q, const GridParams &g,
                  const BwdGeom &bg, const Record *rec, const CellBox *box, const uint32_t *gorder, int64_t n_gauss,
                  const uint32_t *point_off, const float4 *plan_pos, const float2 *ab, float T, float *moments) {
    if (pack == 1)
        hipLaunchKernelGGL((k_backward_gauss<GRID, 1>), dim3(wblocks), dim3(kBwdBlock), 0, s, q, g, bg, rec, box,
                           gorder, n_gauss, point_off, plan_pos, ab, T, moments);
    else if (pack == kPackLarge)
        hipLaunchKernelGGL((k_backward_gauss<GRID, kPackLarge>), dim3(wblocks), dim3(kBwdBlock), 0, s, q, g, bg, rec,
                           box, gorder, n_gauss, point_off, plan_pos, ab, T, moments);
    else
        hipLaunchKernelGGL((k_backward_gauss<GRID, kPack>), dim3(wblocks), dim3(kBwdBlock), 0, s, q, g, bg, rec, box,
                           gorder, n_gauss, point_off, plan_pos, ab, T, moments);
}

}  // namespace

hipError_t launch_count_backward_pairs(const QueryParams &q, const GridParams &g, const BwdGeom &bg,
                                      const Record *rec, const CellBox *box, int64_t n_gauss,
                                      const uint32_t *point_off, unsigned long long *total, hipStream_t s) {
    hipError_t e = fill_u32((uint32_t *)total, 0u, 2, s);
    if (e != hipSuccess || n_gauss <= 0) return e;
    const dim3 grid((uint32_t)((n_gauss + kBlock - 1) / kBlock));
    if (q.kind == 0)
        hipLaunchKernelGGL(k_count_backward_pairs<true>, grid, dim3(kBlock), 0, s, q, g, bg, rec, box, n_gauss,
                           point_off, total);
    else
        hipLaunchKernelGGL(k_count_backward_pairs<false>, grid, dim3(kBlock), 0, s, q, g, bg, rec, box, n_gauss,
                           point_off, total);
    return hipGetLastError();
}

hipError_t launch_backward(const QueryParams &q, const GridParams &g, const BwdGeom &bg, const Record *rec,
                           const CellBox *box, const uint32_t *gorder, int64_t n_gauss, int64_t n_pairs,
                           const uint32_t *order, const uint32_t *point_off, const float4 *plan_pos,
                           const float2 *plan_out, const float *value, const float *influence,
                           const float *grad_value, const float *grad_influence, float T,
                           const BackwardBuffers &b, const float *scale, const float *rot, float *d_mean,
                           float *d_scale, float *d_rot, float *d_value, float *d_weight, hipStream_t s) {
    if (n_gauss <= 0) return hipSuccess;
    hipError_t e;
    const bool grid = q.kind == 0;
    const uint32_t gblocks = (uint32_t)((n_gauss + kBlock - 1) / kBlock);
    if (q.n > 0) {
        const uint32_t qblocks = (uint32_t)((q.n + kBlock - 1) / kBlock);
        prof_begin("bwd_stage", s);
        if (grid) {
            hipLaunchKernelGGL(k_stage_grid, dim3(qblocks), dim3(kBlock), 0, s, q.n, value, influence, grad_value,
                               grad_influence, b.ab);
        } else {
            const dim3 pb((uint32_t)((q.n + kBlock * kStageItems - 1) / (kBlock * kStageItems)));
            const bool vec = ((uintptr_t)grad_value % 16 == 0) && ((uintptr_t)grad_influence % 16 == 0);
            hipLaunchKernelGGL(k_pack_cotangents, pb, dim3(kBlock), 0, s, q.n, grad_value, grad_influence, vec,
                               b.cot);
            hipLaunchKernelGGL(k_stage_plan, dim3(qblocks), dim3(kBlock), 0, s, q.n, order, plan_out, b.cot, b.ab);
        }
        prof_end("bwd_stage", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        // few Gaussians: one per wave, so that they still fill the chip
        const uint32_t pack = n_gauss < kPackMinGauss ? 1u : (n_pairs >= kLargeBoxCells * n_gauss ? kPackLarge : kPack);
        const uint32_t wblocks = (uint32_t)((n_gauss + pack * kBwdWaves - 1) / (pack * kBwdWaves));
        prof_begin("bwd_gauss", s);
        if (grid)
            launch_gauss<true>(pack, wblocks, s, q, g, bg, rec, box, gorder, n_gauss, nullptr, nullptr, b.ab, T,
                               b.moments);
        else
            launch_gauss<false>(pack, wblocks, s, q, g, bg, rec, box, gorder, n_gauss, point_off, plan_pos, b.ab, T,
                                b.moments);
        prof_end("bwd_gauss", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        prof_begin("bwd_zero", s);
        e = fill_f32(b.moments, 0.0f, n_gauss * 12, s);
        prof_end("bwd_zero", s);
        if (e != hipSuccess) return e;
    }
    prof_begin("bwd_finalize", s);
    hipLaunchKernelGGL(k_finalize, dim3(gblocks), dim3(kBlock), 0, s, b.moments, n_gauss, rec, scale, rot, d_mean,
                       d_scale, d_rot, d_value, d_weight);
    prof_end("bwd_finalize", s);
    return hipGetLastError();
}

}  // namespace gs
