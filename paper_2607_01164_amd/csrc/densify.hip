// Weight pruning and sample-error densification on the device
// (include/gs_train.h): Sec. 4.2.1, with false negatives taking priority
// (Sec. 4.2.2).
//
// The ranking is one stable radix sort of a 32-bit key per sample: for an
// eligible sample (in the volume, with a position) the key is
// (false negative << 31 | bits of the float32 error) + 1, whose unsigned
// order is the rank order because a non-negative float's bits order like the
// float; ineligible samples get 0. Sorting the complement ascending puts the
// largest key first and keeps equal keys in sample order. Pruning is a scan
// of the keep flags; a one-block kernel sizes the result; the kept
// Gaussians are scattered to their new slots and the new ones written after
// them. No atomics.
#include "../../include/gs_train.h"
#include "internal.h"

namespace gs {
namespace {

constexpr int kKeyItems = 8;
constexpr int64_t kKeyChunk = (int64_t)kBlock * kKeyItems;
constexpr int kPlanThreads = 1024;

struct DensifyInfo {
    long long n_keep, k, n_out, n_eligible;
};

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
int64_t key_blocks(int64_t nq) { return (nq + kKeyChunk - 1) / kKeyChunk; }

template <typename T>
__device__ __forceinline__ T wsum(T x) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

// Block sum in a fixed order, valid in thread 0.
template <int NT, typename T>
__device__ __forceinline__ T bsum(T x, T *lds) {
    constexpr int kW = NT / kWave;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    x = wsum(x);
    if (lane == 0) lds[wid] = x;
    __syncthreads();
    T r = 0;
    if (wid == 0) r = wsum(lane < kW ? lds[lane] : (T)0);
    __syncthreads();
    return r;
}

__device__ __forceinline__ bool query_has_position(const QueryParams &q, uint32_t pid) {
    if (q.kind == 2 || q.kind == 0 || (q.kind == 3 && !q.voxel_ids)) return true;
    const uint64_t nvox = (uint64_t)(uint32_t)q.dims[0] * (uint32_t)q.dims[1] * (uint32_t)q.dims[2];
    return (uint64_t)q.voxel_ids[pid] < nvox;
}

__global__ __launch_bounds__(kBlock) void k_rank_keys(QueryParams q, const float *value, const float *influence,
                                                      const float *target, const uint8_t *defined, float tau,
                                                      uint32_t *keys, uint32_t *vals, uint32_t *elig_part) {
    __shared__ uint32_t lds[kWavesPerBlock];
    uint32_t ne = 0;
#pragma unroll
    for (int j = 0; j < kKeyItems; ++j) {
        const int64_t i = (int64_t)blockIdx.x * kKeyChunk + (int64_t)j * kBlock + threadIdx.x;
        if (i < q.n) {
            const bool elig = (defined ? defined[i] != 0 : true) && query_has_position(q, (uint32_t)i);
            const float I = influence[i];
            const float e = fabsf(value[i] - target[i]);
            const uint32_t fn = I > tau ? 0u : 1u;
            const uint32_t key = elig ? ((fn << 31) | __float_as_uint(e)) + 1u : 0u;
            keys[i] = ~key;
            vals[i] = (uint32_t)i;
            ne += elig ? 1u : 0u;
        }
    }
    ne = bsum<kBlock>(ne, lds);
    if (threadIdx.x == 0) elig_part[blockIdx.x] = ne;
}

__global__ __launch_bounds__(kBlock) void k_keep_flags(int64_t n, const float *weight, float tau2, uint32_t *flags) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i < n) flags[i] = weight[i] >= tau2 ? 1u : 0u;
    else if (i == n) flags[i] = 0u;
}

__global__ __launch_bounds__(kPlanThreads) void k_densify_plan(const uint32_t *keep_pos, int64_t n_in,
                                                               const uint32_t *elig_part, int64_t nparts,
                                                               long long max_new, long long capacity,
                                                               DensifyInfo *info, long long *n_out) {
    __shared__ unsigned long long lds[kPlanThreads / kWave];
    unsigned long long ne = 0;
    for (int64_t b = threadIdx.x; b < nparts; b += kPlanThreads) ne += elig_part[b];
    ne = bsum<kPlanThreads>(ne, lds);
    if (threadIdx.x == 0) {
        DensifyInfo d;
        d.n_keep = (long long)keep_pos[n_in];
        d.n_eligible = (long long)ne;
        long long k = 0;
        if (d.n_keep <= capacity) {
            k = max_new;
            if (capacity - d.n_keep < k) k = capacity - d.n_keep;
            if (d.n_eligible < k) k = d.n_eligible;
            if (k < 0) k = 0;
        }
        d.k = k;
        d.n_out = d.n_keep + k;
        *info = d;
        *n_out = d.n_out;
    }
}

__global__ __launch_bounds__(kBlock) void k_gather_kept(int64_t n_in, const float *weight, float tau2,
                                                        const uint32_t *keep_pos, long long capacity,
                                                        gs_params in, gs_params out, int32_t *source) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_in || !(weight[i] >= tau2)) return;
    const int64_t d = (int64_t)keep_pos[i];
    if (d >= capacity) return;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        out.mean[3 * d + a] = in.mean[3 * i + a];
        out.log_scale[3 * d + a] = in.log_scale[3 * i + a];
    }
#pragma unroll
    for (int a = 0; a < 4; ++a) out.rot[4 * d + a] = in.rot[4 * i + a];
    out.value_logit[d] = in.value_logit[i];
    out.weight_logit[d] = in.weight_logit[i];
    source[d] = (int32_t)i;
}

__global__ __launch_bounds__(kBlock) void k_spawn(QueryParams q, GridParams g, const uint32_t *ranked,
                                                  const DensifyInfo *info, const float *target, float new_log_scale,
                                                  float new_weight_logit, gs_params out, int32_t *source) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const DensifyInfo d = *info;
    if (j >= d.k) return;
    const uint32_t s = ranked[j];
    const int64_t o = d.n_keep + j;
    float px, py, pz;
    bool valid;
    query_position(q, g, s, px, py, pz, valid);
    out.mean[3 * o] = px;
    out.mean[3 * o + 1] = py;
    out.mean[3 * o + 2] = pz;
#pragma unroll
    for (int a = 0; a < 3; ++a) out.log_scale[3 * o + a] = new_log_scale;
    out.rot[4 * o] = 1.0f;
    out.rot[4 * o + 1] = 0.0f;
    out.rot[4 * o + 2] = 0.0f;
    out.rot[4 * o + 3] = 0.0f;
    // the value of the new Gaussian is the sample's target, as a logit
    const double ylo = 1.0 / 1048576.0, yhi = 1.0 - 1.0 / 1048576.0;
    double y = (double)target[s];
    y = y < ylo ? ylo : (y > yhi ? yhi : y);
    out.value_logit[o] = (float)log(y / (1.0 - y));
    out.weight_logit[o] = new_weight_logit;
    source[o] = -1 - (int32_t)s;
}

struct DensifyWork {
    uint32_t *keys, *vals, *keys2, *vals2;
    char *radix;
    uint32_t *flags, *keep_pos;
    char *scan;
    uint32_t *elig_part;
    DensifyInfo *info;
    long long *n_out;
    size_t bytes;
};

DensifyWork densify_layout(void *base, int64_t n_in, int64_t nq) {
    DensifyWork w{};
    char *b = (char *)base;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *p = b ? b + off : nullptr;
        off = al256(off + bytes);
        return p;
    };
    const size_t mq = (size_t)(nq > 0 ? nq : 1);
    w.keys = (uint32_t *)take(4 * mq);
    w.vals = (uint32_t *)take(4 * mq);
    w.keys2 = (uint32_t *)take(4 * mq);
    w.vals2 = (uint32_t *)take(4 * mq);
    w.radix = take(radix_work_bytes((int64_t)mq, 32));
    w.flags = (uint32_t *)take(4 * (size_t)(n_in + 1));
    w.keep_pos = (uint32_t *)take(4 * (size_t)(n_in + 1));
    w.scan = take(scan_work_bytes(n_in + 1, 4));
    w.elig_part = (uint32_t *)take(4 * (size_t)(key_blocks(nq) > 0 ? key_blocks(nq) : 1));
    w.info = (DensifyInfo *)take(sizeof(DensifyInfo));
    w.n_out = (long long *)take(sizeof(long long));
    w.bytes = off;
    return w;
}

}  // namespace

size_t densify_work_bytes(int64_t n_in, int64_t nq) { return densify_layout(nullptr, n_in, nq).bytes; }

hipError_t launch_densify(const gs_params &in, int64_t n_in, const float *weight, float tau2, const QueryParams &q,
                          const GridParams &g, const float *value, const float *influence, const float *target,
                          const uint8_t *defined, float tau, float new_log_scale, float new_weight_logit,
                          int64_t max_new, int64_t capacity, const gs_params &out, int32_t *source, void *work,
                          long long **n_out_dev, hipStream_t s) {
    const DensifyWork w = densify_layout(work, n_in, q.n);
    *n_out_dev = w.n_out;
    hipError_t e;
    const uint32_t *ranked = w.vals;
    const int64_t nkb = key_blocks(q.n);
    if (q.n > 0) {
        prof_begin("rank_keys", s);
        hipLaunchKernelGGL(k_rank_keys, dim3((uint32_t)nkb), dim3(kBlock), 0, s, q, value, influence, target, defined,
                           tau, w.keys, w.vals, w.elig_part);
        prof_end("rank_keys", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = radix_sort_pairs(w.keys, w.vals, w.keys2, w.vals2, q.n, 32, w.radix, s, false)) != hipSuccess)
            return e;
        ranked = (radix_passes(32) & 1) ? w.vals2 : w.vals;
    }
    prof_begin("keep_flags", s);
    hipLaunchKernelGGL(k_keep_flags, dim3((uint32_t)((n_in + 1 + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, n_in,
                       weight, tau2, w.flags);
    prof_end("keep_flags", s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = exclusive_scan_u32(w.flags, w.keep_pos, n_in + 1, w.scan, s)) != hipSuccess) return e;
    prof_begin("densify_plan", s);
    hipLaunchKernelGGL(k_densify_plan, dim3(1), dim3(kPlanThreads), 0, s, w.keep_pos, n_in, w.elig_part,
                       q.n > 0 ? nkb : (int64_t)0, (long long)max_new, (long long)capacity, w.info, w.n_out);
    prof_end("densify_plan", s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (n_in > 0) {
        prof_begin("gather_kept", s);
        hipLaunchKernelGGL(k_gather_kept, dim3((uint32_t)((n_in + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, n_in,
                           weight, tau2, w.keep_pos, (long long)capacity, in, out, source);
        prof_end("gather_kept", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    int64_t kmax = max_new < capacity ? max_new : capacity;
    kmax = kmax < q.n ? kmax : q.n;
    if (kmax > 0) {
        prof_begin("spawn", s);
        hipLaunchKernelGGL(k_spawn, dim3((uint32_t)((kmax + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, q, g, ranked,
                           w.info, target, new_log_scale, new_weight_logit, out, source);
        prof_end("spawn", s);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace gs
