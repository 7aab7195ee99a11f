/*
 * gs_train.h - the steps on either side of the sampling path in training
 * (paper Sec. 4.2, Sec. 4.2.2, Sec. 5.2): parameter activations and their
 * derivatives, and the reconstruction, false-negative and false-positive
 * losses with the cotangents they hand to gs_sample_backward. Same library
 * and conventions as gs.h: device pointers the caller owns, work enqueued
 * on the caller's stream, gs_status codes with gs_last_error(), no device
 * memory allocated by the library.
 */
#ifndef GS_TRAIN_H
#define GS_TRAIN_H

#include "gs.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Activations (Sec. 4.2) of n Gaussians, computed in float64 and rounded
 * once to float32:
 *   value[i]  = sigmoid(value_logit[i]),  weight[i] = sigmoid(weight_logit[i])
 *   e = exp(log_scale[i][k]) per axis, then a soft cap on the norm of the
 *   scale vector: scale[i] = e * c tanh(|e| / c) / |e|, with c = scale_cap.
 *   The paper names a soft norm cap (0.02; 0.04 for its smallest models)
 *   without its form; this one keeps the direction of e, keeps |scale|
 *   below c and is e to first order when |e| << c. scale_cap <= 0 (or not
 *   finite) disables the cap: scale = e.
 * Means pass through unchanged and the quaternion is normalised inside the
 * sampler, so neither is touched here. Arrays: log_scale and scale
 * [n][3]; the others [n]. An output may be the same buffer as the input it
 * replaces (log_scale as scale, a logit as its activation); other overlaps
 * are not allowed. 0 <= n < 2^31.
 */
gs_status gs_activate(int64_t n, const float *log_scale, const float *value_logit, const float *weight_logit,
                      float scale_cap, float *scale, float *value, float *weight, hipStream_t stream);

/*
 * Chain rule through gs_activate: from the gradients with respect to the
 * activated scale [n][3], value [n] and weight [n] (gs_sample_backward's
 * d_scale, d_value, d_weight) to those of log_scale, value_logit and
 * weight_logit. Evaluated in float64 and rounded once. Each gradient output
 * may be the same buffer as the gradient input it replaces (d_log_scale as
 * d_scale, and so on).
 */
gs_status gs_activate_backward(int64_t n, const float *log_scale, const float *value_logit,
                               const float *weight_logit, float scale_cap, const float *d_scale,
                               const float *d_value, const float *d_weight, float *d_log_scale,
                               float *d_value_logit, float *d_weight_logit, hipStream_t stream);

/* Loss parameters. tau is the cutoff of the sampler (the model is defined
 * where I > tau); fn_eps is Eq. 4's epsilon (>= 0); fn_lambda and fp_lambda
 * are Eq. 4's and Eq. 5's weights (finite). The paper leaves epsilon and the
 * weights to a per-dataset scan. */
typedef struct gs_loss_params {
    float tau;
    float fn_eps;
    float fn_lambda;
    float fp_lambda;
} gs_loss_params;

/* Loss values of a batch, written to device memory by gs_loss. */
typedef struct gs_loss_terms {
    double l1;        /* mean |Phi - y| over D */
    double fn;        /* Eq. 4 */
    double fp;        /* Eq. 5 */
    double total;     /* l1 + fn + fp */
    int64_t n_defined; /* |D| */
    int64_t n_fn;      /* |D-| */
    int64_t n_fp;      /* |U+| */
    int64_t n;         /* samples in the batch */
} gs_loss_terms;

/* Bytes of loss workspace for a batch of n samples (-1 cast to size_t
 * when n < 0). */
size_t gs_loss_work_bytes(int64_t n);

/*
 * Losses of a batch and their cotangents (Sec. 4.2: L1 reconstruction
 * loss; Eq. 4 false negatives; Eq. 5 false positives). Inputs per sample:
 * the sampler's outputs value = Phi and influence = I ((0, 0) where the
 * model is undefined), the target y, and defined[t] != 0 when the sample
 * lies in the original volume (NULL: every sample does, as for the box of
 * a structured volume). With D the samples in the volume and U the others:
 *   L1  = sum over D of |Phi - y| / |D|
 *   LFN = fn_lambda * sum over D- of ((1 + eps) tau - I) / |D-|,
 *         D- = {d in D : I_d < (1 + eps) tau}
 *   LFP = fp_lambda * sum over U+ of I / |U+|,  U+ = {u in U : I_u >= tau}
 * (an empty set contributes 0), with (1 + eps) tau and every sum in
 * float64. The set sizes are constants of the step, so the cotangents are,
 * where the model is defined (I > tau): grad_value = sign(Phi - y) / |D| on
 * D (0 where Phi = y, and on U); grad_influence = -fn_lambda / |D-| on D-,
 * fp_lambda / |U+| on U+, 0 elsewhere; each factor is the float64 quotient
 * rounded once to float32. Where the model is undefined both are 0: no
 * parameter reaches those outputs (Sec. 4.2.2). Writes *terms (device
 * memory). Counts and cotangents are exact and reproducible; the float64
 * sums are formed in a fixed order for a given n, so repeated calls give
 * identical terms. 0 <= n < 2^31.
 */
gs_status gs_loss(int64_t n, const float *value, const float *influence, const float *target,
                  const uint8_t *defined, const gs_loss_params *params, float *grad_value,
                  float *grad_influence, gs_loss_terms *terms, void *work, size_t work_bytes,
                  hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GS_TRAIN_H */
