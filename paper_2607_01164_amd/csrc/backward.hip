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
// The points of a box come as rows: a run of cells along x at fixed (y, z)
// is contiguous in the plan's cell ordering (for grids, a run of voxels is
// contiguous in the x-fastest layout). The wave splits into groups of W
// lanes, W chosen from the mean row length of the Gaussian; each group walks
// one row with W consecutive lanes, so every load instruction reads a few
// whole cache lines. Gaussians are visited in the spatial order of the
// index (the cell key of their box corner), so the waves resident at one
// time work on one region and find its points in L2.
//
// Per pair the partials are kept as 11 moments in the Gaussian's whitened
// frame u = M (p - mu), M = S^-1 R^T, with c = dL/dQ = -1/2 a dL/da:
//   m1 = sum c u (3), m2 = sum c u u^T (6), dv = sum dL/dPhi a / I,
//   dw = sum dL/da G.
// A finalize kernel turns them into dL/dmu = -2 M^T m1,
// dL/ds_k = -2 m2_kk / s_k, dL/dR_jk = (2 / s_k) sum_m R_jm s_m m2_mk, and
// through R(qhat) and qhat = q / |q| into dL/dq.
// For a defined query with outputs (Phi, I) and cotangents (gPhi, gI):
//   dL/da_i = alpha v_i + beta with alpha = gPhi / I, beta = gI - alpha Phi,
// which a staging kernel computes once per query.
#include "internal.h"

#pragma clang fp contract(off)

namespace gs {

namespace {

constexpr float kNegHalfLog2e = -0.72134752044448170368f;

__device__ __forceinline__ void voxel_pos(uint32_t id, const QueryParams &q, const GridParams &g, float &px, float &py,
                                          float &pz) {
    const uint32_t nx = (uint32_t)q.dims[0], ny = (uint32_t)q.dims[1];
    const uint32_t x = id % nx, t = id / nx, y = t % ny, z = t / ny;
    px = g.lo[0] + ((float)x + 0.5f) * q.vsz[0];
    py = g.lo[1] + ((float)y + 0.5f) * q.vsz[1];
    pz = g.lo[2] + ((float)z + 0.5f) * q.vsz[2];
}

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

// Cotangent staging for ordered queries: pts[k] = (x, y, z, alpha) and
// beta[k] of the k-th query in the plan's cell order.
__global__ __launch_bounds__(kBlock) void k_stage_points(QueryParams q, GridParams g,
                                                         const uint32_t *__restrict__ sorted_keys,
                                                         const uint32_t *__restrict__ order,
                                                         const float *__restrict__ value,
                                                         const float *__restrict__ influence,
                                                         const float *__restrict__ gval, const float *__restrict__ ginf,
                                                         float4 *__restrict__ pts, float *__restrict__ beta) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= q.n) return;
    const uint32_t key = sorted_keys[k];
    const uint32_t pid = order[k];
    float px = 0.0f, py = 0.0f, pz = 0.0f, al = 0.0f, be = 0.0f;
    if (key < (uint32_t)g.ncells && (int64_t)pid < q.n) {
        if (q.kind == 1) {
            voxel_pos(q.voxel_ids[pid], q, g, px, py, pz);
        } else {
            px = q.points[3 * (uint64_t)pid];
            py = q.points[3 * (uint64_t)pid + 1];
            pz = q.points[3 * (uint64_t)pid + 2];
        }
        alpha_beta(value[pid], influence[pid], gval[pid], ginf[pid], al, be);
    }
    pts[k] = make_float4(px, py, pz, al);
    beta[k] = be;
}

__global__ __launch_bounds__(kBlock) void k_stage_grid(int64_t n, const float *__restrict__ value,
                                                       const float *__restrict__ influence,
                                                       const float *__restrict__ gval,
                                                       const float *__restrict__ ginf, float *__restrict__ alpha,
                                                       float *__restrict__ beta) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float al, be;
    alpha_beta(value[i], influence[i], gval[i], ginf[i], al, be);
    alpha[i] = al;
    beta[i] = be;
}

struct Acc {
    float m1[3];
    float m2[6];  // 00 01 02 11 12 22
    float dv, dw;
};

__device__ __forceinline__ void pair_grad(const Record &r, float px, float py, float pz, float al, float be, float T,
                                          Acc &acc) {
    const float dx = px - r.r0.x, dy = py - r.r0.y, dz = pz - r.r0.z;
    const float u0 = fmaf_(r.r1.x, dx, fmaf_(r.r1.y, dy, r.r1.z * dz));
    const float u1 = fmaf_(r.r2.x, dx, fmaf_(r.r2.y, dy, r.r2.z * dz));
    const float u2 = fmaf_(r.r3.x, dx, fmaf_(r.r3.y, dy, r.r3.z * dz));
    const float Q = fmaf_(u0, u0, fmaf_(u1, u1, u2 * u2));
    if (Q <= T) {
        const float G = exp2_hw(Q * kNegHalfLog2e);
        const float a = r.r0.w * G;
        const float dLda = fmaf_(al, r.r1.w, be);
        acc.dv = fmaf_(al, a, acc.dv);
        acc.dw = fmaf_(dLda, G, acc.dw);
        const float c = -0.5f * a * dLda;
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
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
    return __builtin_amdgcn_readlane(wave_incl_sum(x), 63);
}

// lanes per row group for a mean row length
__device__ __forceinline__ uint32_t group_width(uint32_t mean_len) {
    return mean_len <= 4 ? 4u : mean_len <= 8 ? 8u : mean_len <= 20 ? 16u : mean_len <= 40 ? 32u : 64u;
}

template <bool GRID>
__global__ __launch_bounds__(kBlock) void k_backward_gauss(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                           const CellBox *__restrict__ box,
                                                           const uint32_t *__restrict__ gorder, int64_t n_gauss,
                                                           const uint32_t *__restrict__ point_off,
                                                           const float4 *__restrict__ pts,
                                                           const float *__restrict__ alpha,
                                                           const float *__restrict__ beta, float T,
                                                           float *__restrict__ moments) {
    const uint32_t lane = threadIdx.x % kWave;
    const uint64_t w = (uint64_t)xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + threadIdx.x / kWave;
    if (w >= (uint64_t)n_gauss) return;
    const uint32_t gid = __builtin_amdgcn_readfirstlane(((ConstU32 *)gorder)[w]);
    const CellBox b = load_box_uniform(box, gid);
    const Record r = load_record_uniform(rec, gid);
    Acc acc;
#pragma unroll
    for (int k = 0; k < 3; ++k) acc.m1[k] = 0.0f;
#pragma unroll
    for (int k = 0; k < 6; ++k) acc.m2[k] = 0.0f;
    acc.dv = acc.dw = 0.0f;
    if (b.hi.x >= b.lo.x) {
        const uint32_t nx = (uint32_t)(b.hi.x - b.lo.x + 1), ny = (uint32_t)(b.hi.y - b.lo.y + 1),
                       nz = (uint32_t)(b.hi.z - b.lo.z + 1);
        uint32_t rx = 1, ry = 1, rz = 1;
        if (GRID) {
            rx = (uint32_t)(q.dims[0] / g.cells[0]);
            ry = (uint32_t)(q.dims[1] / g.cells[1]);
            rz = (uint32_t)(q.dims[2] / g.cells[2]);
        }
        const uint32_t nry = ny * ry, R = nry * nz * rz;
        const uint32_t vx0 = (uint32_t)b.lo.x * rx;
        for (uint32_t rb = 0; rb < R; rb += kWave) {
            // lane l describes row rb + l: its first element and its length
            const uint32_t row = rb + lane;
            uint32_t start = 0, len = 0, ry_ = 0, rz_ = 0;
            if (row < R) {
                const uint32_t yy = row % nry, zz = row / nry;
                if (GRID) {
                    const uint32_t vy = (uint32_t)b.lo.y * ry + yy, vz = (uint32_t)b.lo.z * rz + zz;
                    start = (uint32_t)q.dims[0] * (vy + (uint32_t)q.dims[1] * vz) + vx0;
                    len = nx * rx;
                    ry_ = vy;
                    rz_ = vz;
                } else {
                    const uint32_t cy = (uint32_t)b.lo.y + yy, cz = (uint32_t)b.lo.z + zz;
                    const uint32_t kbase = (uint32_t)g.cells[0] * (cy + (uint32_t)g.cells[1] * cz);
                    start = point_off[kbase + (uint32_t)b.lo.x];
                    len = point_off[kbase + (uint32_t)b.hi.x + 1] - start;
                }
            }
            const uint32_t nrows = (R - rb) < (uint32_t)kWave ? (R - rb) : (uint32_t)kWave;
            const uint32_t W = group_width((wave_sum_u32(len) + nrows - 1) / nrows);
            const uint32_t G = kWave / W;
            const uint32_t grp = lane / W, t = lane % W;
            for (uint32_t rr = 0; rr < nrows; rr += G) {
                // every lane takes part in the shuffles (a lane reading from an
                // inactive lane would get 0); rows past the end have length 0
                const uint32_t my = rr + grp;
                const uint32_t s_start = __shfl(start, (int)my, 64);
                const uint32_t s_len = __shfl(len, (int)my, 64);
                if (GRID) {
                    const uint32_t s_y = __shfl(ry_, (int)my, 64), s_z = __shfl(rz_, (int)my, 64);
                    const float py = g.lo[1] + ((float)s_y + 0.5f) * q.vsz[1];
                    const float pz = g.lo[2] + ((float)s_z + 0.5f) * q.vsz[2];
                    for (uint32_t c = t; c < s_len; c += W) {
                        const float px = g.lo[0] + ((float)(vx0 + c) + 0.5f) * q.vsz[0];
                        pair_grad(r, px, py, pz, alpha[s_start + c], beta[s_start + c], T, acc);
                    }
                } else {
                    for (uint32_t c = t; c < s_len; c += W) {
                        const float4 p = pts[s_start + c];
                        pair_grad(r, p.x, p.y, p.z, p.w, beta[s_start + c], T, acc);
                    }
                }
            }
        }
    }
    float v[11] = {acc.m1[0], acc.m1[1], acc.m1[2], acc.m2[0], acc.m2[1], acc.m2[2],
                   acc.m2[3], acc.m2[4], acc.m2[5], acc.dv,    acc.dw};
#pragma unroll
    for (int k = 0; k < 11; ++k) {
        const float rsum = row16_sum(v[k]);
        v[k] = (__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, rsum), 0)) +
                __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, rsum), 16))) +
               (__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, rsum), 32)) +
                __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, rsum), 48)));
    }
    if (lane == 0) {
        float4 *m = (float4 *)(moments + (size_t)gid * 12);
        m[0] = make_float4(v[0], v[1], v[2], v[3]);
        m[1] = make_float4(v[4], v[5], v[6], v[7]);
        m[2] = make_float4(v[8], v[9], v[10], 0.0f);
    }
}

__global__ __launch_bounds__(kBlock) void k_finalize(const float *__restrict__ moments, int64_t n,
                                                     const float *__restrict__ scale, const float *__restrict__ rot,
                                                     float *__restrict__ d_mean, float *__restrict__ d_scale,
                                                     float *__restrict__ d_rot, float *__restrict__ d_value,
                                                     float *__restrict__ d_weight) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *m = moments + (size_t)i * 12;
    const float4 ma = *(const float4 *)m, mb = *(const float4 *)(m + 4), mc = *(const float4 *)(m + 8);
    const double m1[3] = {ma.x, ma.y, ma.z};
    const double m2s[6] = {ma.w, mb.x, mb.y, mb.z, mb.w, mc.x};
    const bool any = ma.x != 0.0f || ma.y != 0.0f || ma.z != 0.0f || ma.w != 0.0f || mb.x != 0.0f ||
                     mb.y != 0.0f || mb.z != 0.0f || mb.w != 0.0f || mc.x != 0.0f || mc.y != 0.0f || mc.z != 0.0f;
    double dmu[3] = {0, 0, 0}, ds[3] = {0, 0, 0}, dq[4] = {0, 0, 0, 0};
    if (any) {
        const double s[3] = {scale[3 * i], scale[3 * i + 1], scale[3 * i + 2]};
        const double q[4] = {rot[4 * i], rot[4 * i + 1], rot[4 * i + 2], rot[4 * i + 3]};
        const double qn = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
        const double w = q[0] / qn, x = q[1] / qn, y = q[2] / qn, z = q[3] / qn;
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
        double M2[3][3];
        M2[0][0] = m2s[0];
        M2[0][1] = M2[1][0] = m2s[1];
        M2[0][2] = M2[2][0] = m2s[2];
        M2[1][1] = m2s[3];
        M2[1][2] = M2[2][1] = m2s[4];
        M2[2][2] = m2s[5];
        for (int j = 0; j < 3; ++j) {
            double acc = 0.0;
            for (int k = 0; k < 3; ++k) acc += R[j][k] * m1[k] / s[k];
            dmu[j] = -2.0 * acc;
        }
        for (int k = 0; k < 3; ++k) ds[k] = -2.0 * M2[k][k] / s[k];
        double G[3][3];
        for (int j = 0; j < 3; ++j)
            for (int k = 0; k < 3; ++k) {
                double acc = 0.0;
                for (int mm = 0; mm < 3; ++mm) acc += R[j][mm] * s[mm] * M2[mm][k];
                G[j][k] = 2.0 * acc / s[k];
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
        for (int k = 0; k < 4; ++k) dq[k] = (dqh[k] - qh[k] * dot) / qn;
    }
    for (int j = 0; j < 3; ++j) {
        d_mean[3 * i + j] = (float)dmu[j];
        d_scale[3 * i + j] = (float)ds[j];
    }
    for (int k = 0; k < 4; ++k) d_rot[4 * i + k] = (float)dq[k];
    d_value[i] = mc.y;
    d_weight[i] = mc.z;
}

}  // namespace

hipError_t launch_backward(const QueryParams &q, const GridParams &g, const Record *rec, const CellBox *box,
                           const uint32_t *gorder, int64_t n_gauss, const uint32_t *sorted_keys, const uint32_t *order,
                           const uint32_t *point_off, const float *value, const float *influence,
                           const float *grad_value, const float *grad_influence, float T,
                           const BackwardBuffers &b, const float *mean, const float *scale, const float *rot,
                           float *d_mean, float *d_scale, float *d_rot, float *d_value, float *d_weight,
                           hipStream_t s) {
    (void)mean;
    if (n_gauss <= 0) return hipSuccess;
    hipError_t e;
    const bool grid = q.kind == 0;
    const uint32_t gblocks = (uint32_t)((n_gauss + kBlock - 1) / kBlock);
    if (q.n > 0) {
        const uint32_t qblocks = (uint32_t)((q.n + kBlock - 1) / kBlock);
        prof_begin("bwd_stage", s);
        if (grid)
            hipLaunchKernelGGL(k_stage_grid, dim3(qblocks), dim3(kBlock), 0, s, q.n, value, influence, grad_value,
                               grad_influence, b.alpha, b.beta);
        else
            hipLaunchKernelGGL(k_stage_points, dim3(qblocks), dim3(kBlock), 0, s, q, g, sorted_keys, order, value,
                               influence, grad_value, grad_influence, b.pts, b.beta);
        prof_end("bwd_stage", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const uint32_t wblocks = (uint32_t)((n_gauss + kWavesPerBlock - 1) / kWavesPerBlock);
        prof_begin("bwd_gauss", s);
        if (grid)
            hipLaunchKernelGGL(k_backward_gauss<true>, dim3(wblocks), dim3(kBlock), 0, s, q, g, rec, box, gorder,
                               n_gauss, point_off, b.pts, b.alpha, b.beta, T, b.moments);
        else
            hipLaunchKernelGGL(k_backward_gauss<false>, dim3(wblocks), dim3(kBlock), 0, s, q, g, rec, box, gorder,
                               n_gauss, point_off, b.pts, b.alpha, b.beta, T, b.moments);
        prof_end("bwd_gauss", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        prof_begin("bwd_zero", s);
        e = fill_f32(b.moments, 0.0f, n_gauss * 12, s);
        prof_end("bwd_zero", s);
        if (e != hipSuccess) return e;
    }
    prof_begin("bwd_finalize", s);
    hipLaunchKernelGGL(k_finalize, dim3(gblocks), dim3(kBlock), 0, s, b.moments, n_gauss, scale, rot, d_mean, d_scale,
                       d_rot, d_value, d_weight);
    prof_end("bwd_finalize", s);
    return hipGetLastError();
}

}  // namespace gs
