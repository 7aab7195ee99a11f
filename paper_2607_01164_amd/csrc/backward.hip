// Backward pass (paper Sec. 4.1.4, Fig. 4 D-E; Sec. 5.1.2).
//
// The paper assigns a thread to every (Gaussian, block) intersection, sums
// its Gaussian's partials over the block's cells and issues one atomic add
// per intersection. Here the work is Gaussian-major at a finer grain: a work
// item is (Gaussian, up to 16 rows of its box), one DPP row of 16 lanes per
// item, one lane per row. A row is a run of cells along x, whose query
// points are contiguous in the cell ordering of the plan (or a run of
// voxels along x for grids). Each lane accumulates the Gaussian's partial
// sums over its row in registers, the 16 lanes are reduced with DPP, and one
// lane issues a single set of atomic adds per item.
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
#include "expand.h"
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

__device__ __forceinline__ void alpha_beta(float phi, float inf, float gp, float gi, bool defined, float &al,
                                           float &be) {
    if (defined && inf > 0.0f) {
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
    if (key < (uint32_t)g.ncells) {
        if (q.kind == 1) {
            voxel_pos(q.voxel_ids[pid], q, g, px, py, pz);
        } else {
            px = q.points[3 * (uint64_t)pid];
            py = q.points[3 * (uint64_t)pid + 1];
            pz = q.points[3 * (uint64_t)pid + 2];
        }
        alpha_beta(value[pid], influence[pid], gval[pid], ginf[pid], true, al, be);
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
    alpha_beta(value[i], influence[i], gval[i], ginf[i], true, al, be);
    alpha[i] = al;
    beta[i] = be;
}

// Rows of a Gaussian's box: cell rows (cy, cz) for ordered queries, voxel
// rows (vy, vz) for grids.
__device__ __forceinline__ uint32_t box_rows(const CellBox &b, bool grid, uint32_t ry, uint32_t rz) {
    if (b.hi.x < b.lo.x) return 0u;
    const uint32_t ny = (uint32_t)(b.hi.y - b.lo.y + 1), nz = (uint32_t)(b.hi.z - b.lo.z + 1);
    return grid ? ny * ry * nz * rz : ny * nz;
}

__global__ __launch_bounds__(kBlock) void k_item_counts(const CellBox *__restrict__ box, int64_t n, int grid,
                                                        uint32_t ry, uint32_t rz, uint32_t *__restrict__ item_off) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == n) item_off[n] = 0;
    if (i >= n) return;
    const uint32_t rows = box_rows(box[i], grid != 0, ry, rz);
    item_off[i] = (rows + kRowGroup - 1) / kRowGroup;
}

__global__ __launch_bounds__(kBlock) void k_expand_items(const uint32_t *__restrict__ item_off, int64_t n,
                                                         uint32_t *__restrict__ items, int64_t max_items) {
    __shared__ ExpandShared sh;
    const uint64_t total = item_off[n] < (uint64_t)max_items ? item_off[n] : (uint64_t)max_items;
    const uint64_t tile_begin = (uint64_t)blockIdx.x * kExpandTile;
    if (tile_begin >= total) return;
    const uint64_t rem = total - tile_begin;
    const uint32_t tile_cnt = rem < (uint64_t)kExpandTile ? (uint32_t)rem : (uint32_t)kExpandTile;
    const int64_t gfirst = expand_tile(item_off, n, tile_begin, tile_cnt, sh);
#pragma unroll 2
    for (int i = 0; i < kExpandItems; ++i) {
        const uint32_t slot = (uint32_t)i * kBlock + threadIdx.x;
        if (slot < tile_cnt) items[tile_begin + slot] = (uint32_t)(gfirst + sh.head[slot]);
    }
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

// One wave = 4 items of 16 lanes; blocks of 4 waves = 16 items.
__global__ __launch_bounds__(kBlock) void k_backward_rows(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                          const CellBox *__restrict__ box,
                                                          const uint32_t *__restrict__ item_off, int64_t n_gauss,
                                                          const uint32_t *__restrict__ items,
                                                          const uint32_t *__restrict__ point_off,
                                                          const float4 *__restrict__ pts,
                                                          const float *__restrict__ alpha,
                                                          const float *__restrict__ beta, float T,
                                                          float *__restrict__ moments, int64_t max_items) {
    const uint32_t total = item_off[n_gauss] < (uint64_t)max_items ? item_off[n_gauss] : (uint32_t)max_items;
    const uint32_t lane = threadIdx.x % kWave;
    const uint32_t group = lane / kRowGroup, gl = lane % kRowGroup;
    const uint64_t item = ((uint64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave) * (kWave / kRowGroup) + group;
    const bool active = item < total;
    Acc acc;
#pragma unroll
    for (int k = 0; k < 3; ++k) acc.m1[k] = 0.0f;
#pragma unroll
    for (int k = 0; k < 6; ++k) acc.m2[k] = 0.0f;
    acc.dv = acc.dw = 0.0f;
    uint32_t gid = 0;
    if (active) {
        gid = items[item];
        const uint32_t chunk = (uint32_t)item - item_off[gid];
        const uint32_t row = chunk * kRowGroup + gl;
        const CellBox b = box[gid];
        const Record r = rec[gid];
        const bool grid = q.kind == 0;
        if (grid) {
            const uint32_t rx = (uint32_t)(q.dims[0] / g.cells[0]);
            const uint32_t ry = (uint32_t)(q.dims[1] / g.cells[1]);
            const uint32_t rz = (uint32_t)(q.dims[2] / g.cells[2]);
            const uint32_t nvy = (uint32_t)(b.hi.y - b.lo.y + 1) * ry;
            const uint32_t nvz = (uint32_t)(b.hi.z - b.lo.z + 1) * rz;
            if (row < nvy * nvz) {
                const uint32_t vy = (uint32_t)b.lo.y * ry + row % nvy;
                const uint32_t vz = (uint32_t)b.lo.z * rz + row / nvy;
                const uint32_t vx0 = (uint32_t)b.lo.x * rx, vx1 = (uint32_t)(b.hi.x + 1) * rx;
                const float py = g.lo[1] + ((float)vy + 0.5f) * q.vsz[1];
                const float pz = g.lo[2] + ((float)vz + 0.5f) * q.vsz[2];
                const uint64_t rowbase = (uint64_t)q.dims[0] * ((uint64_t)vy + (uint64_t)q.dims[1] * vz);
                for (uint32_t vx = vx0; vx < vx1; ++vx) {
                    const float px = g.lo[0] + ((float)vx + 0.5f) * q.vsz[0];
                    const uint64_t idx = rowbase + vx;
                    pair_grad(r, px, py, pz, alpha[idx], beta[idx], T, acc);
                }
            }
        } else {
            const uint32_t ny = (uint32_t)(b.hi.y - b.lo.y + 1), nz = (uint32_t)(b.hi.z - b.lo.z + 1);
            if (row < ny * nz) {
                const uint32_t cy = (uint32_t)b.lo.y + row % ny;
                const uint32_t cz = (uint32_t)b.lo.z + row / ny;
                const uint64_t kbase = (uint64_t)g.cells[0] * ((uint64_t)cy + (uint64_t)g.cells[1] * cz);
                const uint32_t a0 = point_off[kbase + (uint32_t)b.lo.x];
                const uint32_t a1 = point_off[kbase + (uint32_t)b.hi.x + 1];
                for (uint32_t k = a0; k < a1; ++k) {
                    const float4 p = pts[k];
                    pair_grad(r, p.x, p.y, p.z, p.w, beta[k], T, acc);
                }
            }
        }
    }
    // reduce each group's 16 lanes (every lane of the wave takes part)
    float v[11] = {acc.m1[0], acc.m1[1], acc.m1[2], acc.m2[0], acc.m2[1], acc.m2[2],
                   acc.m2[3], acc.m2[4], acc.m2[5], acc.dv,    acc.dw};
#pragma unroll
    for (int k = 0; k < 11; ++k) v[k] = row16_sum(v[k]);
    if (active && gl == 0) {
        float *m = moments + (size_t)gid * 12;
#pragma unroll
        for (int k = 0; k < 11; ++k)
            if (v[k] != 0.0f) atomicAdd(m + k, v[k]);
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
                           int64_t n_gauss, const uint32_t *sorted_keys, const uint32_t *order,
                           const uint32_t *point_off, const float *value, const float *influence,
                           const float *grad_value, const float *grad_influence, float T,
                           const BackwardBuffers &b, const float *mean, const float *scale, const float *rot,
                           float *d_mean, float *d_scale, float *d_rot, float *d_value, float *d_weight,
                           hipStream_t s) {
    (void)mean;
    if (n_gauss <= 0) return hipSuccess;
    hipError_t e;
    const bool grid = q.kind == 0;
    const uint32_t gblocks = (uint32_t)((n_gauss + 1 + kBlock - 1) / kBlock);
    prof_begin("bwd_zero", s);
    e = fill_f32(b.moments, 0.0f, n_gauss * 12, s);
    prof_end("bwd_zero", s);
    if (e != hipSuccess) return e;
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
        const uint32_t ry = grid ? (uint32_t)(q.dims[1] / g.cells[1]) : 1u;
        const uint32_t rz = grid ? (uint32_t)(q.dims[2] / g.cells[2]) : 1u;
        prof_begin("bwd_items", s);
        hipLaunchKernelGGL(k_item_counts, dim3(gblocks), dim3(kBlock), 0, s, box, n_gauss, grid ? 1 : 0, ry, rz,
                           b.item_off);
        prof_end("bwd_items", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = exclusive_scan_u32(b.item_off, b.item_off, n_gauss + 1, b.scan_work, s)) != hipSuccess) return e;
        if (b.max_items > 0) {
            const uint32_t eblocks = (uint32_t)((b.max_items + kExpandTile - 1) / kExpandTile);
            prof_begin("bwd_expand", s);
            hipLaunchKernelGGL(k_expand_items, dim3(eblocks), dim3(kBlock), 0, s, b.item_off, n_gauss, b.items,
                               b.max_items);
            prof_end("bwd_expand", s);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            const int64_t items_per_block = (int64_t)kWavesPerBlock * (kWave / kRowGroup);
            const uint32_t rblocks = (uint32_t)((b.max_items + items_per_block - 1) / items_per_block);
            prof_begin("bwd_rows", s);
            hipLaunchKernelGGL(k_backward_rows, dim3(rblocks), dim3(kBlock), 0, s, q, g, rec, box, b.item_off,
                               n_gauss, b.items, point_off, b.pts, b.alpha, b.beta, T, b.moments, b.max_items);
            prof_end("bwd_rows", s);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    prof_begin("bwd_finalize", s);
    hipLaunchKernelGGL(k_finalize, dim3(gblocks), dim3(kBlock), 0, s, b.moments, n_gauss, scale, rot, d_mean, d_scale,
                       d_rot, d_value, d_weight);
    prof_end("bwd_finalize", s);
    return hipGetLastError();
}

}  // namespace gs
