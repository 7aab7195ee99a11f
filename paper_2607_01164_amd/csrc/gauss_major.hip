// Gaussian-major forward sampler: the paper's unstructured design
// (Sec. 5.1.2, Fig. 6 B) on this library's point index, kept as a variant of
// gs_sample for comparing the two ways of pairing Gaussians with points.
//
// The paper gives every Gaussian a warp that traverses a BVH over the
// sample positions with the Gaussian's box; its threads evaluate disjoint
// leaf samples and add each contribution to the sample's (V, I) with
// atomics, and a last pass divides V by I. Here the point index is the
// plan's cell ordering (the same one gs_sample builds): the points of a run
// of cells along x are contiguous, so a Gaussian's box (or its trimmed row
// spans) is a list of contiguous point ranges. One wave per Gaussian walks
// them, 64 rows at a time concatenated and 64 points per step, tests every
// point against the cutoff, and adds w G and w v G of each contributing
// pair to per-point float64 accumulators with atomic adds; a final pass
// forms (Phi, I) in float64 and rounds them once. Gaussians are taken in
// the index's spatial order, so concurrently running waves hit nearby
// points in L2.
//
// Sums formed by atomics have no fixed order, so the outputs are not
// bit-reproducible from run to run; the float64 sums keep them within
// float32 rounding of each other.
#include "internal.h"

#pragma clang fp contract(off)

namespace gs {
namespace {


__device__ __forceinline__ float eval_pair(const Record &r, float4 p, float T) {
    const float Q = record_q(r, p.x, p.y, p.z);
    return Q <= T ? r.f0.w * exp2_hw(-Q) : 0.0f;
}

// Position of every query in plan order (the walk below reads them
// contiguously); queries outside the domain sit in the outside bucket,
// which no Gaussian visits.
__global__ __launch_bounds__(kBlock) void k_plan_positions(QueryParams q, GridParams g, const uint32_t *order,
                                                           float4 *pos, double *acc) {
    const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (k >= q.n) return;
    float px, py, pz;
    bool valid;
    query_position(q, g, order[k], px, py, pz, valid);
    pos[k] = make_float4(px, py, pz, 0.0f);
    acc[2 * k] = 0.0;
    acc[2 * k + 1] = 0.0;
}

__global__ __launch_bounds__(kBlock) void k_forward_gauss(GridParams g, BwdGeom bg, const Record *__restrict__ rec,
                                                          const CellBox *__restrict__ box,
                                                          const uint32_t *__restrict__ gorder, int64_t n_gauss,
                                                          const uint32_t *__restrict__ point_off,
                                                          const float4 *__restrict__ pos, float T,
                                                          double *__restrict__ acc) {
    const uint32_t lane = threadIdx.x % kWave;
    const uint64_t w = (uint64_t)xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + threadIdx.x / kWave;
    if (w >= (uint64_t)n_gauss) return;
    const uint32_t gid = __builtin_amdgcn_readfirstlane(gorder[w]);
    const CellBox bx = load_box_uniform(box, gid);
    if (bx.hi.x < bx.lo.x) return;
    const Record r = load_record_uniform(rec, gid);
    const float v = r.f2.w;
    const uint32_t nx = (uint32_t)(bx.hi.x - bx.lo.x + 1), ny = (uint32_t)(bx.hi.y - bx.lo.y + 1);
    const uint32_t R = ny * (uint32_t)(bx.hi.z - bx.lo.z + 1);
    for (uint32_t rb = 0; rb < R; rb += kWave) {
        // lane l: row rb + l of the box, its first point and length: the
        // quarters of its cells the record's cutoff can reach
        const uint32_t row = rb + lane;
        uint32_t start = 0, len = 0;
        if (row < R) {
            const uint32_t zz = row / ny, yy = row - zz * ny;
            len = plan_row(r, (uint32_t)bx.lo.x, nx, (uint32_t)bx.lo.y + yy, (uint32_t)bx.lo.z + zz, g, bg, point_off,
                           start);
        }
        const uint32_t nrows = R - rb < (uint32_t)kWave ? R - rb : (uint32_t)kWave;
        const uint32_t incl = wave_incl_sum(len);
        const uint32_t E = __builtin_amdgcn_readlane(incl, kWave - 1);
        const uint32_t rbeg = incl - len;    // first element of row l in the concatenation
        const uint32_t kofs = start - rbeg;  // element e of row l is point e + kofs
        for (uint32_t e0 = 0; e0 < E; e0 += kWave) {
            // rows starting at or before e0 are a prefix of the lanes (rbeg
            // rises with the lane); the last of them holds element e0
            const uint32_t j0 = (uint32_t)__popcll(mask_le_u(rbeg, e0)) - 1u;
            const uint32_t e = e0 + lane;
            uint32_t ko = __builtin_amdgcn_readlane(kofs, j0);
            // rows starting inside the window, in row order (an empty row is
            // overridden by the next)
            uint64_t inw = mask_lt_u(lane, nrows) & mask_lt_u(rbeg - e0 - 1u, (uint32_t)kWave - 1u);
            while (inw != 0) {
                const uint32_t j = (uint32_t)__builtin_ctzll(inw);
                inw &= inw - 1;
                ko = e >= __builtin_amdgcn_readlane(rbeg, j) ? __builtin_amdgcn_readlane(kofs, j) : ko;
            }
            if (e < E) {
                const uint32_t k = e + ko;
                const float a = eval_pair(r, pos[k], T);
                if (a > 0.0f) {
                    unsafeAtomicAdd(acc + 2 * (size_t)k, (double)a);
                    unsafeAtomicAdd(acc + 2 * (size_t)k + 1, (double)(a * v));
                }
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_finish_gauss_major(int64_t n, const uint32_t *order, const double *acc,
                                                               float tau, float *out_v, float *out_i,
                                                               float2 *plan_out) {
    const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (k >= n) return;
    const double I = acc[2 * k], V = acc[2 * k + 1];
    const float i32 = (float)I;
    const bool def = i32 > tau;
    const float phi = def ? (float)(V / I) : 0.0f, inf = def ? i32 : 0.0f;
    const uint32_t pid = order[k];
    out_v[pid] = phi;
    out_i[pid] = inf;
    plan_out[k] = make_float2(phi, inf);
}

}  // namespace

size_t gauss_major_work_bytes(int64_t nq) { return (size_t)(nq > 0 ? nq : 1) * 2 * sizeof(double); }

hipError_t launch_sample_gauss_major(const QueryParams &q, const GridParams &g, const BwdGeom &bg, const Record *rec,
                                     const CellBox *box, const uint32_t *gorder,
                                     int64_t n_gauss, const uint32_t *order, const uint32_t *point_off, float T,
                                     float tau, float *out_v, float *out_i, const PlanResults &pr, void *work,
                                     hipStream_t s) {
    if (q.n <= 0) return hipSuccess;
    double *acc = (double *)work;
    const uint32_t nb = (uint32_t)((q.n + kBlock - 1) / kBlock);
    prof_begin("gm_positions", s);
    hipLaunchKernelGGL(k_plan_positions, dim3(nb), dim3(kBlock), 0, s, q, g, order, pr.pos, acc);
    prof_end("gm_positions", s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n_gauss > 0) {
        prof_begin("gm_forward", s);
        hipLaunchKernelGGL(k_forward_gauss, dim3((uint32_t)((n_gauss + kWavesPerBlock - 1) / kWavesPerBlock)),
                           dim3(kBlock), 0, s, g, bg, rec, box, gorder, n_gauss, point_off, pr.pos, T, acc);
        prof_end("gm_forward", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    prof_begin("gm_finish", s);
    hipLaunchKernelGGL(k_finish_gauss_major, dim3(nb), dim3(kBlock), 0, s, q.n, order, acc, tau, out_v, out_i,
                       pr.out);
    prof_end("gm_finish", s);
    return hipGetLastError();
}

}  // namespace gs
