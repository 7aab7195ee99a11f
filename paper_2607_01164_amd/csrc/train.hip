// Training epilogue on the device (include/gs_train.h): the activations of
// Sec. 4.2 and their derivatives, and the L1 (Sec. 4.2), false-negative
// (Eq. 4) and false-positive (Eq. 5) losses with the cotangents they hand to
// the sampler's backward.
//
// Both steps are elementwise and bound by HBM traffic, so the arithmetic is
// float64 (free here) and every float32 result is rounded once. The loss is
// a deterministic three-launch reduction: per-block partial sums over a
// fixed partition of the batch, one block that combines them in a fixed
// order and forms the cotangent factors, and an elementwise pass that writes
// the cotangents. No atomics.
#include "../../include/gs_train.h"
#include "internal.h"

namespace gs {
namespace {

constexpr int kLossItems = 8;                       // samples per thread per chunk
constexpr int64_t kLossChunk = (int64_t)kBlock * kLossItems;
constexpr int kLossMaxBlocks = 1024;
constexpr int kFinishThreads = 1024;

struct LossPart {
    double l1, fn, fp;
    unsigned long long nd, nfn, nfp;
};

// Cotangent factors formed by the finishing block: 1/|D|, -lambda_FN/|D-|,
// lambda_FP/|U+| (0 for an empty set).
struct LossScales {
    float g1, gfn, gfp, pad;
};

int64_t loss_chunks(int64_t n) { return (n + kLossChunk - 1) / kLossChunk; }
int loss_blocks(int64_t n) {
    const int64_t c = loss_chunks(n);
    return (int)(c < kLossMaxBlocks ? (c > 0 ? c : 1) : kLossMaxBlocks);
}
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The soft cap's factor g(n) = c tanh(n/c) / n and g'(n) / n. Below
// t = n/c = 1e-4, g = 1 - t^2/3 to float64 accuracy, and g'(n)/n takes its
// limit -2/(3 c^2): the term it enters is itself O(t^2) relative to the
// g dL/ds term, so the neglected O(t^2) part is below float64 rounding.
// Above, the closed form's cancellation in sech^2 - g is of relative size
// 1e-16/t^2, again scaled by t^2 where it enters.
__device__ __forceinline__ void soft_cap(double n, double c, double &g, double &dgn) {
    const double t = n / c;
    if (t < 1e-4) {
        g = 1.0 - t * t * (1.0 / 3.0);
        dgn = -2.0 / (3.0 * c * c);
        return;
    }
    const double th = tanh(t);
    g = th / t;
    dgn = ((1.0 - th * th) - g) / (n * n);
}

__device__ __forceinline__ double sigmoid_d(double x) { return 1.0 / (1.0 + exp(-x)); }

// sigmoid'(x) = e / (1 + e)^2 with e = exp(-|x|): no cancellation at either tail.
__device__ __forceinline__ double sigmoid_grad_d(double x) {
    const double e = exp(-fabs(x));
    const double d = 1.0 + e;
    return e / (d * d);
}

__global__ __launch_bounds__(kBlock) void k_activate(int64_t n, const float *log_scale, const float *value_logit,
                                                     const float *weight_logit, double cap, float *scale,
                                                     float *value, float *weight) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    const double e0 = exp((double)log_scale[3 * i]);
    const double e1 = exp((double)log_scale[3 * i + 1]);
    const double e2 = exp((double)log_scale[3 * i + 2]);
    const double vl = (double)value_logit[i], wl = (double)weight_logit[i];
    double g = 1.0, dgn = 0.0;
    if (cap > 0.0) soft_cap(sqrt(e0 * e0 + e1 * e1 + e2 * e2), cap, g, dgn);
    scale[3 * i] = (float)(e0 * g);
    scale[3 * i + 1] = (float)(e1 * g);
    scale[3 * i + 2] = (float)(e2 * g);
    value[i] = (float)sigmoid_d(vl);
    weight[i] = (float)sigmoid_d(wl);
}

__global__ __launch_bounds__(kBlock) void k_activate_backward(int64_t n, const float *log_scale,
                                                              const float *value_logit, const float *weight_logit,
                                                              double cap, const float *d_scale, const float *d_value,
                                                              const float *d_weight, float *d_log_scale,
                                                              float *d_value_logit, float *d_weight_logit) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    const double e0 = exp((double)log_scale[3 * i]);
    const double e1 = exp((double)log_scale[3 * i + 1]);
    const double e2 = exp((double)log_scale[3 * i + 2]);
    const double s0 = (double)d_scale[3 * i], s1 = (double)d_scale[3 * i + 1], s2 = (double)d_scale[3 * i + 2];
    const double dv = (double)d_value[i], dw = (double)d_weight[i];
    const double vl = (double)value_logit[i], wl = (double)weight_logit[i];
    double g = 1.0, dgn = 0.0;
    if (cap > 0.0) soft_cap(sqrt(e0 * e0 + e1 * e1 + e2 * e2), cap, g, dgn);
    // s = e g(|e|): dL/de = g dL/ds + (dL/ds . e) g'(|e|) e / |e|; dL/dlog e = dL/de * e
    const double k = (s0 * e0 + s1 * e1 + s2 * e2) * dgn;
    d_log_scale[3 * i] = (float)((g * s0 + k * e0) * e0);
    d_log_scale[3 * i + 1] = (float)((g * s1 + k * e1) * e1);
    d_log_scale[3 * i + 2] = (float)((g * s2 + k * e2) * e2);
    d_value_logit[i] = (float)(dv * sigmoid_grad_d(vl));
    d_weight_logit[i] = (float)(dw * sigmoid_grad_d(wl));
}

template <typename T>
__device__ __forceinline__ T wave_sum_xor(T x) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}


// The six loss sums of a block, reduced together in a fixed order: each
// wave's tree sums, one LDS row per wave, then the first wave sums the rows
// in wave order (one barrier for all six instead of two per sum). The
// result is valid in thread 0.
struct LossSums {
    double l1, fn, fp;
    unsigned long long nd, nfn, nfp;
};

template <int NT>
__device__ __forceinline__ LossSums block_sum_loss(LossSums x, LossSums *lds) {
    constexpr int kW = NT / kWave;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    x.l1 = wave_sum_xor(x.l1);
    x.fn = wave_sum_xor(x.fn);
    x.fp = wave_sum_xor(x.fp);
    x.nd = wave_sum_xor(x.nd);
    x.nfn = wave_sum_xor(x.nfn);
    x.nfp = wave_sum_xor(x.nfp);
    if (lane == 0) lds[wid] = x;
    __syncthreads();
    LossSums r{0.0, 0.0, 0.0, 0ull, 0ull, 0ull};
    if (wid == 0) {
        if (lane < kW) r = lds[lane];
        r.l1 = wave_sum_xor(r.l1);
        r.fn = wave_sum_xor(r.fn);
        r.fp = wave_sum_xor(r.fp);
        r.nd = wave_sum_xor(r.nd);
        r.nfn = wave_sum_xor(r.nfn);
        r.nfp = wave_sum_xor(r.nfp);
    }
    return r;
}

__global__ __launch_bounds__(kBlock) void k_loss_partials(int64_t n, int64_t chunks, const float *value,
                                                          const float *influence, const float *target,
                                                          const uint8_t *defined, float tau, double thr,
                                                          LossPart *part) {
    __shared__ LossSums lds[kBlock / kWave];
    double l1 = 0.0, fn = 0.0, fp = 0.0;
    unsigned nd = 0, nfn = 0, nfp = 0;
    for (int64_t c = blockIdx.x; c < chunks; c += gridDim.x) {
        const int64_t base = c * kLossChunk + threadIdx.x;
        float v[kLossItems], I[kLossItems], y[kLossItems];
        bool ok[kLossItems], d[kLossItems];
#pragma unroll
        for (int j = 0; j < kLossItems; ++j) {
            const int64_t i = base + (int64_t)j * kBlock;
            ok[j] = i < n;
            v[j] = ok[j] ? value[i] : 0.0f;
            I[j] = ok[j] ? influence[i] : 0.0f;
            y[j] = ok[j] ? target[i] : 0.0f;
            d[j] = ok[j] && (defined ? defined[i] != 0 : true);
        }
#pragma unroll
        for (int j = 0; j < kLossItems; ++j) {
            if (!ok[j]) continue;
            if (d[j]) {
                ++nd;
                l1 += fabs((double)v[j] - (double)y[j]);
                if ((double)I[j] < thr) {
                    ++nfn;
                    fn += thr - (double)I[j];
                }
            } else if (I[j] >= tau) {
                ++nfp;
                fp += (double)I[j];
            }
        }
    }
    const LossSums r = block_sum_loss<kBlock>(LossSums{l1, fn, fp, nd, nfn, nfp}, lds);
    if (threadIdx.x == 0) {
        LossPart p;
        p.l1 = r.l1;
        p.fn = r.fn;
        p.fp = r.fp;
        p.nd = r.nd;
        p.nfn = r.nfn;
        p.nfp = r.nfp;
        part[blockIdx.x] = p;
    }
}

__global__ __launch_bounds__(kFinishThreads) void k_loss_finish(int nparts, const LossPart *part, int64_t n,
                                                                 float lambda_fn, float lambda_fp,
                                                                 gs_loss_terms *terms, LossScales *scales) {
    __shared__ LossSums lds[kFinishThreads / kWave];
    const int t = threadIdx.x;
    double l1 = 0.0, fn = 0.0, fp = 0.0;
    unsigned long long nd = 0, nfn = 0, nfp = 0;
    if (t < nparts) {
        const LossPart p = part[t];
        l1 = p.l1;
        fn = p.fn;
        fp = p.fp;
        nd = p.nd;
        nfn = p.nfn;
        nfp = p.nfp;
    }
    const LossSums r = block_sum_loss<kFinishThreads>(LossSums{l1, fn, fp, nd, nfn, nfp}, lds);
    l1 = r.l1;
    fn = r.fn;
    fp = r.fp;
    nd = r.nd;
    nfn = r.nfn;
    nfp = r.nfp;
    if (t == 0) {
        const double dnd = (double)nd, dnfn = (double)nfn, dnfp = (double)nfp;
        gs_loss_terms r;
        r.l1 = nd ? l1 / dnd : 0.0;
        r.fn = nfn ? (double)lambda_fn * fn / dnfn : 0.0;
        r.fp = nfp ? (double)lambda_fp * fp / dnfp : 0.0;
        r.total = r.l1 + r.fn + r.fp;
        r.n_defined = (int64_t)nd;
        r.n_fn = (int64_t)nfn;
        r.n_fp = (int64_t)nfp;
        r.n = n;
        *terms = r;
        LossScales s;
        s.g1 = nd ? (float)(1.0 / dnd) : 0.0f;
        s.gfn = nfn ? (float)(-(double)lambda_fn / dnfn) : 0.0f;
        s.gfp = nfp ? (float)((double)lambda_fp / dnfp) : 0.0f;
        s.pad = 0.0f;
        *scales = s;
    }
}

__global__ __launch_bounds__(kBlock) void k_loss_grads(int64_t n, const float *value, const float *influence,
                                                       const float *target, const uint8_t *defined, float tau,
                                                       double thr, const LossScales *scales, float *grad_value,
                                                       float *grad_influence) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    const LossScales s = *scales;
    const float v = value[i], I = influence[i], y = target[i];
    const bool in_d = defined ? defined[i] != 0 : true;
    float gv = 0.0f, gi = 0.0f;
    if (I > tau) {  // the model is defined at this sample
        if (in_d) {
            gv = v > y ? s.g1 : (v < y ? -s.g1 : 0.0f);
            if ((double)I < thr) gi = s.gfn;
        } else {
            gi = s.gfp;
        }
    }
    grad_value[i] = gv;
    grad_influence[i] = gi;
}

}  // namespace

size_t loss_work_bytes(int64_t n) {
    return align256((size_t)loss_blocks(n) * sizeof(LossPart)) + align256(sizeof(LossScales));
}

hipError_t launch_activate(int64_t n, const float *log_scale, const float *value_logit, const float *weight_logit,
                           double cap, float *scale, float *value, float *weight, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    prof_begin("activate", s);
    hipLaunchKernelGGL(k_activate, dim3((uint32_t)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, n, log_scale,
                       value_logit, weight_logit, cap, scale, value, weight);
    prof_end("activate", s);
    return hipGetLastError();
}

hipError_t launch_activate_backward(int64_t n, const float *log_scale, const float *value_logit,
                                    const float *weight_logit, double cap, const float *d_scale,
                                    const float *d_value, const float *d_weight, float *d_log_scale,
                                    float *d_value_logit, float *d_weight_logit, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    prof_begin("activate_bwd", s);
    hipLaunchKernelGGL(k_activate_backward, dim3((uint32_t)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, n,
                       log_scale, value_logit, weight_logit, cap, d_scale, d_value, d_weight, d_log_scale,
                       d_value_logit, d_weight_logit);
    prof_end("activate_bwd", s);
    return hipGetLastError();
}

hipError_t launch_loss(int64_t n, const float *value, const float *influence, const float *target,
                       const uint8_t *defined, float tau, float eps, float lambda_fn, float lambda_fp,
                       float *grad_value, float *grad_influence, gs_loss_terms *terms, void *work, hipStream_t s) {
    const int nb = loss_blocks(n);
    const int64_t chunks = loss_chunks(n);
    LossPart *part = (LossPart *)work;
    LossScales *scales = (LossScales *)((char *)work + align256((size_t)nb * sizeof(LossPart)));
    const double thr = (1.0 + (double)eps) * (double)tau;
    if (n > 0) {
        prof_begin("loss_partials", s);
        hipLaunchKernelGGL(k_loss_partials, dim3((uint32_t)nb), dim3(kBlock), 0, s, n, chunks, value, influence,
                           target, defined, tau, thr, part);
        prof_end("loss_partials", s);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    prof_begin("loss_finish", s);
    hipLaunchKernelGGL(k_loss_finish, dim3(1), dim3(kFinishThreads), 0, s, n > 0 ? nb : 0, part, n, lambda_fn,
                       lambda_fp, terms, scales);
    prof_end("loss_finish", s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n <= 0) return e;
    prof_begin("loss_grads", s);
    hipLaunchKernelGGL(k_loss_grads, dim3((uint32_t)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, n, value,
                       influence, target, defined, tau, thr, scales, grad_value, grad_influence);
    prof_end("loss_grads", s);
    return hipGetLastError();
}

}  // namespace gs
