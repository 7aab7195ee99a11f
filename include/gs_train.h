/*
 * gs_train.h - the steps on either side of the sampling path in training
 * (paper Sec. 4.2, Sec. 4.2.1, Sec. 4.2.2, Sec. 5.2): parameter activations
 * and their derivatives, the reconstruction, false-negative and
 * false-positive losses with the cotangents they hand to
 * gs_sample_backward, and weight pruning with sample-error densification. Same library
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

/* Free parameters of a set of Gaussians, before the activations: means
 * [n][3], log-scales [n][3], quaternions [n][4] (w, x, y, z), value logits
 * [n] and weight logits [n]. */
typedef struct gs_params {
    float *mean;
    float *log_scale;
    float *rot;
    float *value_logit;
    float *weight_logit;
} gs_params;

/* Densification and pruning settings (Sec. 4.2.1). */
typedef struct gs_densify_params {
    float prune_weight;     /* tau_2: a Gaussian whose activated weight is below it is removed (0.005) */
    float tau;              /* the sampler's cutoff: the model is undefined where I <= tau */
    float new_log_scale;    /* log of the isotropic standard deviation of a new Gaussian */
    float new_weight_logit; /* weight logit of a new Gaussian (logit(0.01) for the initial weight 0.01) */
    int64_t max_new;        /* k: new Gaussians at most (the paper uses 1/5 of the final count) */
} gs_densify_params;

/* Bytes of densification workspace for n_in Gaussians and a query (-1 cast
 * to size_t for a malformed query or count). */
size_t gs_densify_work_bytes(int64_t n_in, const gs_query *query);

/*
 * Weight pruning and sample-error densification (Sec. 4.2.1, with false
 * negatives first, Sec. 4.2.2), run after a forward pass and gs_loss.
 *   Pruning: Gaussian i of the input set is kept when weight[i] (its
 *   activated weight, float32, as gs_activate wrote it) >= prune_weight;
 *   the kept Gaussians keep their order.
 *   Ranking: sample t of the query (the outputs value, influence of
 *   gs_sample, the targets, and the volume flags as for gs_loss, NULL: all
 *   in the volume) is eligible when it lies in the volume and has a
 *   position (a voxel id past the grid has none). Eligible samples are
 *   ranked false negatives (I <= tau) first, then by the float32 error
 *   |value - target| from largest to smallest, ties by increasing t.
 *   Spawning: k = min(max_new, capacity - kept, eligible) new Gaussians at
 *   the positions (as gs_sample computes them, over the box of domain) of
 *   the first k ranked samples, set up as at initialisation: log-scale
 *   new_log_scale on every axis, rotation (1, 0, 0, 0), value logit
 *   log(y / (1 - y)) of the sample's target clamped to [2^-20, 1 - 2^-20]
 *   (float64, rounded once), weight logit new_weight_logit.
 * Output (out, arrays of capacity Gaussians, not overlapping in): the kept
 * Gaussians, then the new ones in rank order; source[j] = the input index
 * of output j, or -1 - t for a new Gaussian made at sample t, so that other
 * per-Gaussian state (optimiser moments) can be carried over with the same
 * map. Waits on the stream once and sets *n_out (host) to the output count.
 * When the kept Gaussians alone exceed the capacity, returns
 * GS_ERR_CAPACITY with *n_out = the kept count and out unspecified (nothing
 * is written past the capacity). Rebuild the index (gs_build_index) on the
 * new set before sampling it. 0 <= n_in, capacity < 2^31.
 */
gs_status gs_densify(const gs_params *in, int64_t n_in, const float *weight, const gs_grid *domain,
                     const gs_query *query, const float *value, const float *influence, const float *target,
                     const uint8_t *defined, const gs_densify_params *params, const gs_params *out,
                     int64_t capacity, int32_t *source, int64_t *n_out, void *work, size_t work_bytes,
                     hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GS_TRAIN_H */
