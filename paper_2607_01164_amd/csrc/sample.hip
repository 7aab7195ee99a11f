// Forward sampling (paper Eq. 2 with the cutoff test of Sec. 4.1.1 and the
// definedness rule of Sec. 4.1.3).
//
// Grid queries (Sec. 4.1.3, Fig. 4 C): one wavefront per (cell, 64 voxels of
// the cell); every lane is a voxel and all lanes walk the cell's Gaussian
// list together, so the list entries and the 64-byte Gaussian records are
// wave-uniform and come through scalar loads into SGPRs rather than through
// shared-memory batches.
//
// Voxel-list and point queries (Sec. 5.1.2): the queries are first ordered
// by cell (query_keys + radix sort, kept in the plan); a wavefront takes 64
// consecutive ordered queries. When they share one cell the wave takes the
// same scalar path; otherwise every lane walks its own cell's list with
// vector loads, which neighbouring lanes of one cell share.
#include "internal.h"

#pragma clang fp contract(off)

namespace gs {

namespace {

// -1/2 log2(e): G = exp(-Q/2) = 2^(Q * kNegHalfLog2e)
constexpr float kNegHalfLog2e = -0.72134752044448170368f;

__device__ __forceinline__ void accumulate(const Record &r, float px, float py, float pz, float T, float &I,
                                           float &V) {
    const float dx = px - r.r0.x, dy = py - r.r0.y, dz = pz - r.r0.z;
    const float u0 = fmaf_(r.r1.x, dx, fmaf_(r.r1.y, dy, r.r1.z * dz));
    const float u1 = fmaf_(r.r2.x, dx, fmaf_(r.r2.y, dy, r.r2.z * dz));
    const float u2 = fmaf_(r.r3.x, dx, fmaf_(r.r3.y, dy, r.r3.z * dz));
    const float Q = fmaf_(u0, u0, fmaf_(u1, u1, u2 * u2));
    if (Q <= T) {
        const float a = r.r0.w * exp2_hw(Q * kNegHalfLog2e);
        I += a;
        V = fmaf_(a, r.r1.w, V);
    }
}

// Walk a wave-uniform list [j0, j1): list entries and records through the
// scalar path.
__device__ __forceinline__ void walk_uniform(const Record *rec, const uint32_t *gids, uint32_t j0, uint32_t j1,
                                             float px, float py, float pz, float T, float &I, float &V) {
    ConstU32 *cg = (ConstU32 *)gids;
    uint32_t j = j0;
    for (; j + 2 <= j1; j += 2) {
        const uint32_t g0 = __builtin_amdgcn_readfirstlane(cg[j]);
        const uint32_t g1 = __builtin_amdgcn_readfirstlane(cg[j + 1]);
        const Record a = load_record_uniform(rec, g0);
        const Record b = load_record_uniform(rec, g1);
        accumulate(a, px, py, pz, T, I, V);
        accumulate(b, px, py, pz, T, I, V);
    }
    if (j < j1) {
        const uint32_t g0 = __builtin_amdgcn_readfirstlane(cg[j]);
        const Record a = load_record_uniform(rec, g0);
        accumulate(a, px, py, pz, T, I, V);
    }
}

// Walk a per-lane list with vector loads.
__device__ __forceinline__ void walk_lane(const Record *__restrict__ rec, const uint32_t *__restrict__ gids, uint32_t j0,
                                          uint32_t j1, float px, float py, float pz, float T, float &I, float &V) {
    for (uint32_t j = j0; j < j1; ++j) {
        const uint32_t gg = gids[j];
        const Record r = rec[gg];
        accumulate(r, px, py, pz, T, I, V);
    }
}

__device__ __forceinline__ float voxel_center(int32_t i, float lo, float vs) { return lo + ((float)i + 0.5f) * vs; }

__global__ __launch_bounds__(kBlock) void k_sample_grid(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                        const uint32_t *__restrict__ gids,
                                                        const uint32_t *__restrict__ cell_off, float T, float tau,
                                                        float *__restrict__ out_v, float *__restrict__ out_i) {
    const uint32_t rx = (uint32_t)(q.dims[0] / g.cells[0]);
    const uint32_t ry = (uint32_t)(q.dims[1] / g.cells[1]);
    const uint32_t rz = (uint32_t)(q.dims[2] / g.cells[2]);
    const uint32_t vpc = rx * ry * rz;
    const uint32_t wpc = (vpc + kWave - 1) / kWave;
    const uint32_t lane = threadIdx.x % kWave;
    const uint64_t wave_id =
        (uint64_t)xcd_block(blockIdx.x, gridDim.x) * kWavesPerBlock + threadIdx.x / kWave;
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
    walk_uniform(rec, gids, j0, j1, px, py, pz, T, I, V);
    if (local < vpc) {
        const uint64_t idx = (uint64_t)vx + (uint64_t)q.dims[0] * ((uint64_t)vy + (uint64_t)q.dims[1] * (uint64_t)vz);
        const bool def = I > tau;
        out_v[idx] = def ? V / I : 0.0f;
        out_i[idx] = def ? I : 0.0f;
    }
}

__device__ __forceinline__ void query_position(const QueryParams &q, const GridParams &g, uint32_t pid, float &px,
                                               float &py, float &pz, bool &valid) {
    valid = true;
    if (q.kind == 1) {
        const uint32_t id = q.voxel_ids[pid];
        const uint32_t nx = (uint32_t)q.dims[0], ny = (uint32_t)q.dims[1], nz = (uint32_t)q.dims[2];
        const uint64_t nvox = (uint64_t)nx * ny * nz;
        if ((uint64_t)id >= nvox) {
            valid = false;
            px = py = pz = 0.0f;
            return;
        }
        const uint32_t x = id % nx, t = id / nx, y = t % ny, z = t / ny;
        px = voxel_center((int32_t)x, g.lo[0], q.vsz[0]);
        py = voxel_center((int32_t)y, g.lo[1], q.vsz[1]);
        pz = voxel_center((int32_t)z, g.lo[2], q.vsz[2]);
    } else {
        px = q.points[3 * (uint64_t)pid];
        py = q.points[3 * (uint64_t)pid + 1];
        pz = q.points[3 * (uint64_t)pid + 2];
    }
}

__global__ __launch_bounds__(kBlock) void k_query_keys(QueryParams q, GridParams g, uint32_t *__restrict__ keys,
                                                       uint32_t *__restrict__ ids) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= q.n) return;
    float p[3];
    bool valid;
    query_position(q, g, (uint32_t)i, p[0], p[1], p[2], valid);
    uint32_t key = (uint32_t)g.ncells;
    if (valid) {
        bool inside = true;
        int64_t c[3];
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            inside = inside && (p[j] >= g.lo[j]) && (p[j] <= g.hi[j]);
            const float t = (p[j] - g.lo[j]) * g.invc[j];
            int64_t ci = (int64_t)floorf(t);
            ci = ci < 0 ? 0 : ci;
            ci = ci > g.cells[j] - 1 ? g.cells[j] - 1 : ci;
            c[j] = ci;
        }
        if (inside) key = (uint32_t)(c[0] + (int64_t)g.cells[0] * (c[1] + (int64_t)g.cells[1] * c[2]));
    }
    keys[i] = key;
    ids[i] = (uint32_t)i;
}

__global__ __launch_bounds__(kBlock) void k_sample_points(QueryParams q, GridParams g, const Record *__restrict__ rec,
                                                          const uint32_t *__restrict__ gids,
                                                          const uint32_t *__restrict__ cell_off,
                                                          const uint32_t *__restrict__ sorted_keys,
                                                          const uint32_t *__restrict__ order, float T, float tau,
                                                          float *__restrict__ out_v, float *__restrict__ out_i) {
    const int64_t k = (int64_t)xcd_block(blockIdx.x, gridDim.x) * kBlock + threadIdx.x;
    const bool active = k < q.n;
    const uint32_t ncells = (uint32_t)g.ncells;
    const uint32_t pid = active ? order[k] : 0u;
    const uint32_t key = (active && (int64_t)pid < q.n) ? sorted_keys[k] : ncells;
    float px = 0.0f, py = 0.0f, pz = 0.0f;
    bool valid = false;
    if (active && key < ncells) query_position(q, g, pid, px, py, pz, valid);
    const bool work = active && key < ncells && valid;
    float I = 0.0f, V = 0.0f;
    // all working lanes in one cell: walk the shared list through the scalar path
    const uint64_t wmask = __ballot(work);
    const uint32_t kfirst = wmask ? __shfl(key, (int)__builtin_ctzll(wmask), 64) : 0u;
    const bool uniform = wmask != 0 && __ballot(work && key != kfirst) == 0;
    if (uniform) {
        const uint32_t kk = __builtin_amdgcn_readfirstlane(kfirst);
        const uint32_t j0 = __builtin_amdgcn_readfirstlane(cell_off[kk]);
        const uint32_t j1 = __builtin_amdgcn_readfirstlane(cell_off[kk + 1]);
        walk_uniform(rec, gids, j0, j1, px, py, pz, T, I, V);
    } else if (work) {
        walk_lane(rec, gids, cell_off[key], cell_off[key + 1], px, py, pz, T, I, V);
    }
    if (active && (int64_t)pid < q.n) {
        const bool def = work && I > tau;
        out_v[pid] = def ? V / I : 0.0f;
        out_i[pid] = def ? I : 0.0f;
    }
}

}  // namespace

hipError_t launch_query_keys(const QueryParams &q, const GridParams &g, uint32_t *keys, uint32_t *ids,
                             hipStream_t s) {
    if (q.n <= 0) return hipSuccess;
    prof_begin("query_keys", s);
    hipLaunchKernelGGL(k_query_keys, dim3((uint32_t)((q.n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, q, g, keys,
                       ids);
    prof_end("query_keys", s);
    return hipGetLastError();
}

hipError_t launch_sample_grid(const QueryParams &q, const GridParams &g, const Record *rec, const uint32_t *gids,
                              const uint32_t *cell_off, float T, float tau, float *out_v, float *out_i,
                              hipStream_t s) {
    const int64_t vpc = (int64_t)(q.dims[0] / g.cells[0]) * (q.dims[1] / g.cells[1]) * (q.dims[2] / g.cells[2]);
    const int64_t wpc = (vpc + kWave - 1) / kWave;
    const int64_t waves = g.ncells * wpc;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks <= 0) return hipSuccess;
    prof_begin("sample_grid", s);
    hipLaunchKernelGGL(k_sample_grid, dim3((uint32_t)blocks), dim3(kBlock), 0, s, q, g, rec, gids, cell_off, T, tau,
                       out_v, out_i);
    prof_end("sample_grid", s);
    return hipGetLastError();
}

hipError_t launch_sample_points(const QueryParams &q, const GridParams &g, const Record *rec, const uint32_t *gids,
                                const uint32_t *cell_off, const uint32_t *sorted_keys, const uint32_t *order,
                                float T, float tau, float *out_v, float *out_i, hipStream_t s) {
    if (q.n <= 0) return hipSuccess;
    prof_begin("sample_points", s);
    hipLaunchKernelGGL(k_sample_points, dim3((uint32_t)((q.n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, q, g, rec,
                       gids, cell_off, sorted_keys, order, T, tau, out_v, out_i);
    prof_end("sample_points", s);
    return hipGetLastError();
}

}  // namespace gs
