/*
 * gs.h - point sampling of a learned 3D-Gaussian scalar field (W-VEG) on
 * AMD Instinct MI355X (gfx950), forward and backward.
 *
 * The field (paper Sec. 3.2, Eq. 2 and Eq. 3):
 *   Gaussian i has mean mu_i, per-axis standard deviations s_i, a rotation
 *   given by the quaternion q_i = (w, x, y, z) (normalised inside the library,
 *   Hamilton convention, rotating the Gaussian's local axes into world axes),
 *   a value v_i and a weight w_i.
 *   Q_i(p) = || S_i^-1 R(q_i)^T (p - mu_i) ||^2,  G_i(p) = exp(-Q_i(p) / 2).
 *   Gaussian i intersects p when G_i(p) >= tau (the cutoff of Sec. 4.1.1),
 *   i.e. Q_i(p) <= 2 ln(1/tau). Over the intersecting Gaussians
 *   I(p) = sum w_i G_i(p) and V(p) = sum w_i v_i G_i(p).
 *   A query point is defined when it lies in the closed box of the grid and
 *   I(p) > tau (Sec. 4.1.3); its outputs are then (Phi, I) = (V/I, I), and
 *   (0, 0) otherwise.
 *
 * Conventions for every entry point:
 *   - All array arguments are device pointers to memory the caller allocated
 *     and owns (hipMalloc or a framework allocator). The library allocates no
 *     device memory; the workspaces it needs are passed in, sized by the
 *     *_bytes functions. Workspace pointers must be 256-byte aligned.
 *   - Work is enqueued on the caller's stream and is asynchronous, except that
 *     gs_build_index waits once for the number of Gaussian-cell pairs,
 *     gs_densify (gs_train.h) once for the new Gaussian count, and
 *     gs_backward_pair_count and gs_sample_pair_counts for their counts.
 *   - Errors are reported as gs_status codes; gs_last_error() returns a
 *     message for the calling thread. Nothing throws across this interface.
 *   - Host-side arguments are validated (null pointers, negative counts,
 *     empty or non-finite grids, workspace sizes, query shapes). Device data
 *     is not: a Gaussian with a non-finite parameter, a non-positive scale or
 *     a quaternion whose float32 squared norm is zero or not finite
 *     contributes nothing anywhere; an out-of-range voxel id is a point
 *     outside the domain.
 *   - Parameters are taken after the paper's activations (Sec. 4.2: exp for
 *     scales, sigmoid for values and weights, with any soft cap applied by
 *     the caller); gradients are returned with respect to those same
 *     parameters, and for the quaternion with respect to the raw (not
 *     normalised) input.
 */
#ifndef GS_H
#define GS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gs_status {
    GS_OK = 0,
    GS_ERR_INVALID_ARGUMENT = 1, /* a host-side argument is invalid */
    GS_ERR_CAPACITY = 2,         /* the pair buffers of an index are too small */
    GS_ERR_WORKSPACE = 3,        /* a workspace is too small or misaligned */
    GS_ERR_HIP = 4               /* a HIP runtime call failed */
} gs_status;

/* The Gaussians (Sec. 3.2: mu, S, R, v, w of each W-VEG primitive). */
typedef struct gs_gaussians {
    int64_t n;           /* number of Gaussians, 0 <= n < 2^31 */
    const float *mean;   /* [n][3] */
    const float *scale;  /* [n][3] standard deviations along the local axes */
    const float *rot;    /* [n][4] quaternion (w, x, y, z), any non-zero norm */
    const float *value;  /* [n] */
    const float *weight; /* [n] */
} gs_gaussians;

/* The domain box [lo, hi] (closed) and the grid of index cells over it.
 * Cells play the role of the paper's volume blocks (Sec. 4.1.1, Fig. 4):
 * each cell gets the list of Gaussians whose cutoff box overlaps it. */
typedef struct gs_grid {
    float lo[3];
    float hi[3];
    int32_t cells[3]; /* cells per axis, each > 0, product < 2^31 (< 2^30 for
                         VOXELS, POINTS and JITTER queries, whose sort keys
                         are 4 cell + quarter in 32 bits) */
} gs_grid;

/* A built index. The caller fills the buffer fields; gs_build_index fills
 * the rest. The pair lists are the paper's block intersection lists
 * (Sec. 4.1.2): pairs (cell key, Gaussian id) with
 * key = cx + Cx (cy + Cy cz), ordered by key and, within a key, by
 * increasing Gaussian id; cell_offsets[k] is the number of pairs with
 * key < k, so the list of cell k is [cell_offsets[k], cell_offsets[k+1]). */
typedef struct gs_index {
    /* caller-owned device buffers */
    uint32_t *keys;         /* [capacity] */
    uint32_t *gids;         /* [capacity] */
    uint32_t *cell_offsets; /* [ncells + 1] */
    int64_t capacity;       /* pairs the two buffers above can hold */
    void *work;             /* gs_index_work_bytes() bytes; after the build it
                               holds per-Gaussian records read by gs_sample and
                               gs_sample_backward: keep it unchanged while the
                               index is in use */
    size_t work_bytes;
    /* filled by gs_build_index */
    int64_t n_pairs;  /* number of pairs (also set on GS_ERR_CAPACITY) */
    int64_t n_gauss;  /* Gaussians the index was built from */
    gs_grid grid;     /* copy of the grid */
    float tau;        /* copy of the cutoff */
} gs_index;

/* Query kinds. GRID: every voxel centre of a dims[0] x dims[1] x dims[2]
 * grid spanning the index box, outputs in x-fastest order; dims must be a
 * multiple of the index cells on every axis. VOXELS: the centres of the
 * listed voxel ids (id = x + dims0 (y + dims1 z)) of such a grid (any dims),
 * outputs in list order. POINTS: arbitrary positions, outputs in input
 * order. The centre of voxel (i, j, k) is lo + (i + 1/2) * ((hi - lo) / dims)
 * per axis, in float32 with each operation rounded.
 * JITTER: the training samples of Sec. 4.2.2, one random position inside
 * each listed voxel (every voxel, x fastest, when voxel_ids is NULL; then n
 * must equal the voxel count): query t lies at
 * lo + (i + u) * ((hi - lo) / dims) per axis, with the caller's offsets
 * u = points[t][axis] (drawn in [0, 1) for a position inside the voxel),
 * in float32 with each operation rounded; outputs in list order. A voxel id
 * past the grid gives an undefined output, as for VOXELS. */
enum { GS_QUERY_GRID = 0, GS_QUERY_VOXELS = 1, GS_QUERY_POINTS = 2, GS_QUERY_JITTER = 3 };

typedef struct gs_query {
    int32_t kind;
    int32_t dims[3];            /* GRID, VOXELS, JITTER */
    int64_t n;                  /* VOXELS, POINTS, JITTER: number of queries, < 2^31 */
    const uint32_t *voxel_ids;  /* VOXELS: [n]; JITTER: [n] or NULL (all voxels) */
    const float *points;        /* POINTS: [n][3] positions; JITTER: [n][3] offsets u */
} gs_query;

/* Number of outputs of a query (dims product for GRID, n otherwise), or -1
 * when the query is malformed. */
int64_t gs_query_size(const gs_query *query);

/* Bytes of index workspace for n_gauss Gaussians, a grid and a pair
 * capacity (per-Gaussian records, boxes, row runs and evaluation flags,
 * row records of the large boxes (one per pair of capacity), scan and sort
 * buffers). */
size_t gs_index_work_bytes(int64_t n_gauss, const gs_grid *grid, int64_t capacity);

/*
 * Build the cell index (Sec. 4.1.1 and Sec. 4.1.2, Fig. 4 A-B): per
 * Gaussian, the axis-aligned box of its cutoff ellipsoid Q <= 2 ln(1/tau)
 * in cells, the per-cell intersection lists and their ranges. tau is the
 * paper's tau_1 (0.01 in its evaluation), 0 < tau < 1.
 * Boxes are computed in float32 in one fixed order of operations, so the
 * index is reproducible bit for bit. The half-extent along axis j is
 * r * sqrt(Sigma_jj) with r = sqrt(2 ln(1/tau)) (1 + 2^-10). A box of at
 * most 4096 (y, z) rows lists, in each row, only the run of cells that the
 * enlarged ellipsoid Q <= r^2 can reach over the row's (y, z) slab, bounded
 * in float64: x conditioned on (y, z) is centred on a line through the mean
 * with half-width sqrt((r^2 - Q2) vc), Q2 the (y, z) marginal's quadratic
 * form and vc the conditional variance; the run covers
 * [min centre - wm, max centre + wm] over the slab's corners, with
 * wm = sqrt((r^2 - min Q2) vc), and is empty when min Q2 > r^2. Every cell
 * holding a point with Q <= 2 ln(1/tau) is still listed. Boxes of more than
 * 64 rows or 16 cells a row keep one record per row with cells in the
 * workspace, taken from room for `capacity` records in stretches of the
 * box's row count; a box that finds no room lists every cell of its box.
 * With a capacity of at least the rows of those boxes, the index (and with
 * it every result) is reproducible bit for bit.
 * Waits on the stream once, for the pair count. If it exceeds the capacity,
 * returns GS_ERR_CAPACITY with index->n_pairs set to the count needed and the
 * index left unusable.
 */
gs_status gs_build_index(const gs_gaussians *gauss, const gs_grid *grid, float tau, gs_index *index,
                         hipStream_t stream);

/* Bytes of plan workspace a query needs with an index of this grid (0 for
 * GRID queries; -1 cast to size_t on a malformed query, or for an ordered
 * query on a grid of 2^30 cells or more, which gs_sample rejects with
 * GS_ERR_INVALID_ARGUMENT). */
size_t gs_plan_bytes(const gs_query *query, const gs_grid *grid);

/*
 * Forward sampling (Eq. 2 with the intersection test of Sec. 4.1.1 and the
 * definedness rule of Sec. 4.1.3; Fig. 4 C for grids, Sec. 5.1.2 for
 * unstructured points): writes out_value[t] = Phi and out_influence[t] = I
 * for every query t, (0, 0) where undefined. gauss must be the Gaussians the
 * index was built from, unchanged. For VOXELS and POINTS queries, plan
 * receives the query ordering and, in that order, each query's position and
 * (Phi, I), which gs_sample_backward reuses (the paper reuses its sample BVH
 * the same way, Sec. 5.1.2); GRID queries need none.
 * Deterministic: the same inputs give bit-identical outputs.
 */
gs_status gs_sample(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                    float *out_value, float *out_influence, void *plan, size_t plan_bytes,
                    hipStream_t stream);

/*
 * gs_sample in two parts, so that the query ordering (Sec. 5.1.1's role of
 * the sample BVH), which needs only the queries and the grid, can run on
 * another stream while gs_build_index runs: gs_plan_queries fills the
 * plan's ordering and work items for a query and an index grid (nothing
 * for GRID queries, whose plan may be null); gs_sample_planned then samples
 * as gs_sample does, with a plan that gs_plan_queries filled for the same
 * query and the index's grid, unchanged since (the caller orders the two
 * streams, e.g. with an event). The outputs and the plan's contents equal
 * gs_sample's, bit for bit. Plans follow gs_plan_bytes; errors as gs_sample.
 */
gs_status gs_plan_queries(const gs_query *query, const gs_grid *grid, void *plan, size_t plan_bytes,
                          hipStream_t stream);
gs_status gs_sample_planned(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                            float *out_value, float *out_influence, void *plan, size_t plan_bytes,
                            hipStream_t stream);

/* Bytes of workspace gs_sample_gaussian_major needs for a query (16 per
 * query; -1 cast to size_t for a GRID or malformed query). */
size_t gs_sample_gaussian_major_work_bytes(const gs_query *query);

/*
 * Forward sampling in the paper's Gaussian-major form (Sec. 5.1.2, Fig. 6
 * B), a variant of gs_sample for VOXELS, POINTS and JITTER queries kept for
 * comparing the two ways of pairing Gaussians with points. The queries are
 * ordered by cell as gs_sample orders them; then one wavefront per Gaussian
 * walks the points of its box (each row of cells cut to the quarters of
 * cells the Gaussian's cutoff, enlarged by 2^-7, can reach), tests each
 * against the cutoff and adds w G and w v G to that point's float64 sums
 * with atomic adds; a last pass writes (Phi, I) = (V/I, I) where I > tau
 * and the point lies in the box, (0, 0) elsewhere. The outputs equal
 * gs_sample's up to float32 rounding: the atomic sums have no fixed order,
 * so they are not bit-reproducible between runs. The plan is left as
 * gs_sample leaves it, so gs_sample_backward can follow. work: 256-byte
 * aligned, gs_sample_gaussian_major_work_bytes() bytes.
 */
gs_status gs_sample_gaussian_major(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                                   float *out_value, float *out_influence, void *plan, size_t plan_bytes,
                                   void *work, size_t work_bytes, hipStream_t stream);

/*
 * Bytes of backward workspace for an index (built) and a query: 48 per
 * Gaussian and 8 per query (16 for VOXELS, POINTS and JITTER queries), in
 * 256-byte aligned parts; (size_t)-1 for invalid arguments.
 */
size_t gs_backward_work_bytes(const gs_index *index, const gs_query *query);

/*
 * Backward pass (Sec. 4.1.4, Fig. 4 D-E; Sec. 5.1.2): given the forward
 * outputs (value, influence) of gs_sample for this index, query and plan,
 * and cotangents grad_value = dL/dPhi and grad_influence = dL/dI per query,
 * overwrites the gradients of L with respect to every parameter:
 * d_mean [n][3], d_scale [n][3], d_rot [n][4] (w.r.t. the raw quaternion),
 * d_value [n], d_weight [n]. Undefined queries carry no gradient. The
 * intersecting sets are those of the forward pass (the result is the exact
 * derivative of the smooth piece). For VOXELS and POINTS queries the
 * forward outputs are read from the copy gs_sample left in the plan, so
 * value and influence must be that call's outputs (they are read as given
 * for GRID queries). Every per-Gaussian sum is formed by one wavefront in a
 * fixed order, without atomics: the same inputs give bit-identical results.
 * Each Gaussian's queries are walked in rows along x (rows of voxels for
 * GRID queries, rows of index cells in the plan's order otherwise), each
 * cut to the x-range of the cutoff ellipsoid, enlarged by 2^-7 in Q, over
 * the row's (y, z) extent: to whole voxels, or to quarters of cells.
 */
gs_status gs_sample_backward(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                             const void *plan, size_t plan_bytes, const float *value, const float *influence,
                             const float *grad_value, const float *grad_influence, float *d_mean,
                             float *d_scale, float *d_rot, float *d_value, float *d_weight, void *work,
                             size_t work_bytes, hipStream_t stream);

/*
 * gs_sample_backward for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving or training loops, harnesses that
 * forbid hipMalloc. Same arguments, results and errors as
 * gs_sample_backward (bit-identical outputs), except that its workspace is
 * a static device array of GS_BACKWARD_NOALLOC_MAX_BYTES inside the
 * library instead of a caller buffer: no device memory is allocated or
 * freed. Each GPU the library runs on holds its own copy of that array
 * from the library's load until the process ends. A call whose workspace
 * (gs_backward_work_bytes) would exceed it returns GS_ERR_WORKSPACE. Calls
 * on one GPU share its array, and every call overwrites what the last one
 * left there (nothing in it needs to start cleared): calls that may
 * overlap on one GPU (other streams, other host threads) race and must be
 * ordered by the caller.
 */
#define GS_BACKWARD_NOALLOC_MAX_BYTES ((size_t)64 << 20)
gs_status gs_sample_backward_noalloc(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                                     const void *plan, size_t plan_bytes, const float *value, const float *influence,
                                     const float *grad_value, const float *grad_influence, float *d_mean,
                                     float *d_scale, float *d_rot, float *d_value, float *d_weight,
                                     hipStream_t stream);

/*
 * For measurement: the number of (Gaussian, query) pairs gs_sample_backward
 * tests against the cutoff for this built index, query and plan (the plan
 * a gs_sample call filled; none for GRID queries): per Gaussian, the
 * queries of its rows (see gs_sample_backward), each cut to the row's
 * x-range: whole voxels for GRID queries, quarters of cells along x
 * otherwise. Uses work (gs_backward_work_bytes() bytes, its contents are
 * overwritten) and waits on the stream for the count.
 */
gs_status gs_backward_pair_count(const gs_index *index, const gs_query *query, const void *plan,
                                 size_t plan_bytes, void *work, size_t work_bytes, int64_t *count,
                                 hipStream_t stream);

/*
 * For measurement: the (Gaussian, query) pairs gs_sample tests against the
 * cutoff for this built index and query (*tests: per query, the length of
 * its cell's list; queries outside the domain test none) and how many of
 * them pass it (*contributing: Q <= 2 ln(1/tau) in the samplers' own float32
 * arithmetic, the pairs that enter Eq. 2; the backward's contributing pairs
 * are the same). For VOXELS, POINTS and JITTER queries plan must be the one
 * a gs_sample call on this index and query filled (it reads the query order
 * and positions kept there). Uses work (gs_backward_work_bytes() bytes, its
 * contents are overwritten) and waits on the stream for the counts.
 */
gs_status gs_sample_pair_counts(const gs_index *index, const gs_query *query, const void *plan, size_t plan_bytes,
                                void *work, size_t work_bytes, int64_t *tests, int64_t *contributing,
                                hipStream_t stream);

/* Message describing the last failure on the calling thread ("" if none). */
const char *gs_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int gs_version(void);

/*
 * Kernel timing, for measurement. While enabled, every kernel the library
 * launches is bracketed by HIP events on its stream. gs_profile_read waits
 * for the recorded events and returns, for up to max_entries kernels, their
 * names (pointers into static storage), launch counts and summed durations
 * in milliseconds; the return value is the number of distinct kernels seen.
 * gs_profile_enable(0) stops recording; gs_profile_reset() clears the
 * records. gs_profile_select(name) limits the recording to the kernel of
 * that name (the names gs_profile_read reports); NULL records every kernel.
 * The name is copied. Not thread-safe; meant for one measuring thread.
 */
void gs_profile_enable(int on);
void gs_profile_select(const char *name);
void gs_profile_reset(void);
int gs_profile_read(const char **names, int64_t *counts, double *total_ms, int max_entries);

#ifdef __cplusplus
}
#endif

#endif /* GS_H */
