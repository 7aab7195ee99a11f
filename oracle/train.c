/*
 * CPU oracle for the steps on either side of the sampling path in training:
 * the parameter activations and their derivatives (Sec. 4.2), the
 * reconstruction, false-negative and false-positive losses (Sec. 4.2, Eq. 4,
 * Eq. 5) with the cotangents they hand to the sampler's backward, and
 * sample-error densification with weight pruning (Sec. 4.2.1).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do. It shares no code, header or constant with the GPU path.
 * Arithmetic is float64 on the float32 inputs, in plain loops.
 *
 * Activations (Sec. 4.2). Values and weights are sigmoids of free
 * parameters, v = sigmoid(v'), w = sigmoid(w'). Scales are exponentials,
 * e = exp(s') per axis, followed by a soft cap on the norm of the scale
 * vector: s = e * c tanh(|e| / c) / |e|. The paper names a soft norm cap
 * of 0.02 (0.04 for the smallest models) without its form; this reading
 * keeps the direction of e, bounds |s| below c, and is e to first order
 * when |e| << c. A cap c <= 0 means no cap, s = e. Means pass through, and
 * the quaternion is normalised inside the sampler.
 *
 * Losses, over a batch of n samples with model outputs (Phi, I) (the
 * sampler's, (0, 0) where the model is undefined, i.e. I <= tau), targets y
 * and a flag telling whether the sample is defined in the original volume:
 *   D   = samples defined in the volume, U = the others;
 *   L1  = sum over D of |Phi - y| / |D|                        (Sec. 4.2)
 *   D-  = {d in D : I_d < (1 + eps) tau},
 *   LFN = lambda_FN * sum over D- of ((1 + eps) tau - I_d) / |D-|   (Eq. 4)
 *   U+  = {u in U : I_u >= tau},
 *   LFP = lambda_FP * sum over U+ of I_u / |U+|                  (Eq. 5)
 *   L   = L1 + LFN + LFP; an empty set contributes 0.
 * The set sizes are constants of the step (they change only where a sample
 * crosses a threshold), so the cotangents are, at samples where the model
 * is defined: dL/dPhi = sign(Phi - y) / |D| on D (0 where Phi = y), and
 * dL/dI = -lambda_FN / |D-| on D-, +lambda_FP / |U+| on U+. Where the model
 * is undefined no parameter reaches the outputs (Sec. 4.2.2: training cannot
 * move a false negative directly), and both cotangents are 0.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORC_OK 0
#define ORC_ERR_ARG 1

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* c tanh(n / c) / n, the factor of the soft cap, and its derivative in n
 * divided by n. For t = n / c below 1e-2 both come from their Taylor series
 * (tanh(t) / t = 1 - t^2/3 + 2 t^4/15 - ..., and
 * (sech^2(t) - tanh(t)/t) / t^2 = -2/3 + 8 t^2/15 - 34 t^4/105 + ...), which
 * avoids the cancellation of the closed form there. */
static void cap_factor(double n, double c, double *g, double *dg_over_n)
{
    const double t = n / c;
    if (t < 1e-2) {
        const double t2 = t * t;
        *g = 1.0 - t2 / 3.0 + 2.0 * t2 * t2 / 15.0;
        *dg_over_n = (-2.0 / 3.0 + 8.0 * t2 / 15.0 - 34.0 * t2 * t2 / 105.0) / (c * c);
        return;
    }
    const double th = tanh(t), sech2 = 1.0 - th * th;
    *g = th / t;
    *dg_over_n = (sech2 - th / t) / (n * n);
}

/* Activations of n Gaussians: scale [n][3], value [n], weight [n]. */
int orc_activate(int64_t n, const double *log_scale, const double *value_logit, const double *weight_logit,
                 double cap, double *scale, double *value, double *weight)
{
    if (n < 0) return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; ++i) {
        double e[3], nrm2 = 0.0;
        for (int k = 0; k < 3; ++k) {
            e[k] = exp(log_scale[3 * i + k]);
            nrm2 += e[k] * e[k];
        }
        double g = 1.0, dgn = 0.0;
        if (cap > 0.0) cap_factor(sqrt(nrm2), cap, &g, &dgn);
        for (int k = 0; k < 3; ++k) scale[3 * i + k] = e[k] * g;
        value[i] = sigmoid(value_logit[i]);
        weight[i] = sigmoid(weight_logit[i]);
    }
    return ORC_OK;
}

/* Chain rule through the activations: from the gradients with respect to
 * the activated scale, value and weight to those of the free parameters.
 * With s_k = e_k g(|e|): dL/de_j = g dL/ds_j + (sum_k dL/ds_k e_k) g'(|e|)
 * e_j / |e|, and dL/ds'_j = dL/de_j e_j; sigmoid'(x) = sigmoid(x) sigmoid(-x). */
int orc_activate_backward(int64_t n, const double *log_scale, const double *value_logit,
                          const double *weight_logit, double cap, const double *d_scale, const double *d_value,
                          const double *d_weight, double *d_log_scale, double *d_value_logit,
                          double *d_weight_logit)
{
    if (n < 0) return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; ++i) {
        double e[3], nrm2 = 0.0, dot = 0.0;
        for (int k = 0; k < 3; ++k) {
            e[k] = exp(log_scale[3 * i + k]);
            nrm2 += e[k] * e[k];
            dot += d_scale[3 * i + k] * e[k];
        }
        double g = 1.0, dgn = 0.0;
        if (cap > 0.0) cap_factor(sqrt(nrm2), cap, &g, &dgn);
        for (int k = 0; k < 3; ++k) {
            const double dLde = g * d_scale[3 * i + k] + dot * dgn * e[k];
            d_log_scale[3 * i + k] = dLde * e[k];
        }
        /* sigmoid'(x) = sigmoid(x) sigmoid(-x), which unlike
         * sigmoid(x) (1 - sigmoid(x)) does not round to 0 for large x */
        d_value_logit[i] = d_value[i] * (sigmoid(value_logit[i]) * sigmoid(-value_logit[i]));
        d_weight_logit[i] = d_weight[i] * (sigmoid(weight_logit[i]) * sigmoid(-weight_logit[i]));
    }
    return ORC_OK;
}

/* Losses and cotangents of a batch. defined may be NULL (every sample is
 * defined in the volume, as for a structured volume's box). Writes
 * terms = {L1, LFN, LFP, L}, counts = {|D|, |D-|, |U+|} and the cotangents
 * in float32 (each the float64 quotient rounded once). */
int orc_loss(int64_t n, const float *value, const float *influence, const float *target, const uint8_t *defined,
             float tau, float eps, float lambda_fn, float lambda_fp, double *terms, int64_t *counts,
             float *grad_value, float *grad_influence)
{
    if (n < 0) return ORC_ERR_ARG;
    const double t = (double)tau;
    const double thr = (1.0 + (double)eps) * t;
    double l1 = 0.0, fn = 0.0, fp = 0.0;
    int64_t nd = 0, nfn = 0, nfp = 0;
    for (int64_t i = 0; i < n; ++i) {
        const int in_d = defined ? defined[i] != 0 : 1;
        const double I = (double)influence[i];
        if (in_d) {
            ++nd;
            l1 += fabs((double)value[i] - (double)target[i]);
            if (I < thr) {
                ++nfn;
                fn += thr - I;
            }
        } else if (I >= t) {
            ++nfp;
            fp += I;
        }
    }
    terms[0] = nd ? l1 / (double)nd : 0.0;
    terms[1] = nfn ? (double)lambda_fn * fn / (double)nfn : 0.0;
    terms[2] = nfp ? (double)lambda_fp * fp / (double)nfp : 0.0;
    terms[3] = terms[0] + terms[1] + terms[2];
    counts[0] = nd;
    counts[1] = nfn;
    counts[2] = nfp;
    const float g1 = nd ? (float)(1.0 / (double)nd) : 0.0f;
    const float gfn = nfn ? (float)(-(double)lambda_fn / (double)nfn) : 0.0f;
    const float gfp = nfp ? (float)((double)lambda_fp / (double)nfp) : 0.0f;
    for (int64_t i = 0; i < n; ++i) {
        const int in_d = defined ? defined[i] != 0 : 1;
        const double I = (double)influence[i];
        float gv = 0.0f, gi = 0.0f;
        if (I > t) { /* the model is defined here */
            if (in_d) {
                const double d = (double)value[i] - (double)target[i];
                gv = d > 0.0 ? g1 : (d < 0.0 ? -g1 : 0.0f);
                if (I < thr) gi = gfn;
            } else {
                gi = gfp; /* I > tau implies I >= tau */
            }
        }
        grad_value[i] = gv;
        grad_influence[i] = gi;
    }
    return ORC_OK;
}

/*
 * Sample-error densification and weight pruning (Sec. 4.2.1, with the false
 * negatives of Sec. 4.2.2 taking priority).
 *   Pruning: a Gaussian is kept when its (activated, float32) weight is at
 *   least tau2; the kept ones stay in their order.
 *   Ranking: a sample is eligible when it lies in the volume (defined flag,
 *   or every sample when the flags are absent) and has a position (valid).
 *   It is a false negative when the model is undefined there (I <= tau).
 *   Eligible samples are ranked false negatives first, then by the float32
 *   error |Phi - y| from largest to smallest, ties by increasing index.
 *   Spawning: k = min(max_new, capacity - kept, eligible) new Gaussians, one
 *   at the position of each of the first k ranked samples, set up as at
 *   initialisation: isotropic log-scale new_log_scale, identity rotation,
 *   the sample's target as value (logit of y clamped to [2^-20, 1 - 2^-20]),
 *   weight logit new_weight_logit.
 * Output: the kept Gaussians' parameters in order, then the new ones in rank
 * order; source[j] = the input index of output j, or -1 - s for a new
 * Gaussian made at sample s. Returns the output count, or -1 - kept when
 * the kept Gaussians alone exceed the capacity (nothing written then).
 */
typedef struct {
    int fn;
    float err;
    int64_t idx;
} ranked;

static int rank_cmp(const void *pa, const void *pb)
{
    const ranked *a = (const ranked *)pa, *b = (const ranked *)pb;
    if (a->fn != b->fn) return a->fn > b->fn ? -1 : 1;
    if (a->err != b->err) return a->err > b->err ? -1 : 1;
    return a->idx < b->idx ? -1 : (a->idx > b->idx ? 1 : 0);
}

int64_t orc_densify(int64_t n_in, const float *mean, const float *log_scale, const float *rot,
                    const float *value_logit, const float *weight_logit, const float *weight, float tau2,
                    int64_t nq, const float *pos, const uint8_t *valid, const float *value, const float *influence,
                    const float *target, const uint8_t *defined, float tau, float new_log_scale,
                    float new_weight_logit, int64_t max_new, int64_t capacity, float *o_mean, float *o_log_scale,
                    float *o_rot, float *o_value_logit, float *o_weight_logit, int32_t *source)
{
    int64_t kept = 0;
    for (int64_t i = 0; i < n_in; ++i)
        if (weight[i] >= tau2) ++kept;
    if (kept > capacity) return -1 - kept;
    ranked *r = (ranked *)malloc(sizeof(ranked) * (size_t)(nq > 0 ? nq : 1));
    if (!r) return -1 - kept;
    int64_t ne = 0;
    for (int64_t s = 0; s < nq; ++s) {
        const int in_d = defined ? defined[s] != 0 : 1;
        if (!in_d || !valid[s]) continue;
        r[ne].fn = !(influence[s] > tau);
        r[ne].err = fabsf(value[s] - target[s]);
        r[ne].idx = s;
        ++ne;
    }
    qsort(r, (size_t)ne, sizeof(ranked), rank_cmp);
    int64_t k = max_new;
    if (capacity - kept < k) k = capacity - kept;
    if (ne < k) k = ne;
    if (k < 0) k = 0;
    int64_t j = 0;
    for (int64_t i = 0; i < n_in; ++i) {
        if (!(weight[i] >= tau2)) continue;
        for (int a = 0; a < 3; ++a) {
            o_mean[3 * j + a] = mean[3 * i + a];
            o_log_scale[3 * j + a] = log_scale[3 * i + a];
        }
        for (int a = 0; a < 4; ++a) o_rot[4 * j + a] = rot[4 * i + a];
        o_value_logit[j] = value_logit[i];
        o_weight_logit[j] = weight_logit[i];
        source[j] = (int32_t)i;
        ++j;
    }
    const double ylo = 1.0 / 1048576.0, yhi = 1.0 - 1.0 / 1048576.0;
    for (int64_t t = 0; t < k; ++t, ++j) {
        const int64_t s = r[t].idx;
        for (int a = 0; a < 3; ++a) {
            o_mean[3 * j + a] = pos[3 * s + a];
            o_log_scale[3 * j + a] = new_log_scale;
        }
        o_rot[4 * j] = 1.0f;
        o_rot[4 * j + 1] = o_rot[4 * j + 2] = o_rot[4 * j + 3] = 0.0f;
        double y = (double)target[s];
        y = y < ylo ? ylo : (y > yhi ? yhi : y);
        o_value_logit[j] = (float)log(y / (1.0 - y));
        o_weight_logit[j] = new_weight_logit;
        source[j] = (int32_t)(-1 - s);
    }
    free(r);
    return j;
}
