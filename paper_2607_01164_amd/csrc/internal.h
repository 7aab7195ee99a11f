// Internal declarations shared by the HIP translation units of the library:
// the per-Gaussian record layout, small wave/block primitives, and the host
// launchers the C-ABI layer calls. Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace gs {

constexpr int kWave = 64;
constexpr int kBlock = 256;             // threads per workgroup for most kernels
constexpr int kWavesPerBlock = kBlock / kWave;

// Per-Gaussian evaluation record, 48 bytes, written by the preprocess:
//   f0 = (mu_x, mu_y, mu_z, w)
//   f1 = (U00, U01, U02, w v)    U = kRecScale L, L upper triangular with
//   f2 = (U11, U12, U22, v)      L^T L = R S^-2 R^T (the inverse covariance)
// so that |U (p - mu)|^2 = Q' = Q log2(e) / 2 and G = exp(-Q/2) = 2^-Q'; the
// forward adds w G and (w v) G with one FMA each (w v rounded once); the
// cutoff G >= tau reads Q' <= log2(1/tau) (record_T). L, the Cholesky
// factor of the inverse covariance, takes 6 products and sums where
// M = S^-1 R^T takes 9, and three 16-byte quarters where M takes four; its
// float32 rounding bounds Q as M's does (L and M have the same 2-norm).
// Formed in float64, scaled, and rounded once. Invalid Gaussians get zeros,
// an empty box, and appear in no cell list.
struct alignas(16) Record {
    float4 f0, f1, f2;
};
constexpr int kRecordQuads = 3;  // 16-byte quarters of a Record

// sqrt(log2(e) / 2), the factor of the record's U
constexpr double kRecScale = 0.84932180028801904272;

// Q' = |U (p - mu)|^2 = Q log2(e) / 2 in float32, as the grid sampler,
// the forward's sparse and row-layout cells, the Gaussian-major forward and
// the pair counter form it (the dense cells' walk forms the same Q' from
// offsets to the cell's centre, see offset_planes).
__device__ __forceinline__ float record_q(const Record &r, float px, float py, float pz) {
    const float dx = px - r.f0.x, dy = py - r.f0.y, dz = pz - r.f0.z;
    const float u0 = __builtin_fmaf(r.f1.x, dx, __builtin_fmaf(r.f1.y, dy, r.f1.z * dz));
    const float u1 = __builtin_fmaf(r.f2.x, dy, r.f2.y * dz);
    const float u2 = r.f2.z * dz;
    return __builtin_fmaf(u0, u0, __builtin_fmaf(u1, u1, u2 * u2));
}

// A record loaded with a wave-uniform address (scalar loads).
__device__ __forceinline__ Record load_record_uniform(const Record *rec, uint32_t g) {
    typedef float f4u __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(4))) const f4u CF4;
    CF4 *p = (CF4 *)rec + kRecordQuads * (size_t)g;
    const f4u a = p[0], b = p[1], c = p[2];
    Record r;
    r.f0 = make_float4(a.x, a.y, a.z, a.w);
    r.f1 = make_float4(b.x, b.y, b.z, b.w);
    r.f2 = make_float4(c.x, c.y, c.z, c.w);
    return r;
}

// Cell box of a Gaussian: (x0, y0, z0, trim) and (x1, y1, z1, nrec),
// inclusive; an empty box has x1 < x0. A trimmed box (trim 1 or 2) lists,
// in each of its (y, z) rows (row r = (y - y0) + ny (z - z0)), only the run
// of cells that a bound of the cutoff ellipsoid (enlarged like the box)
// over the row's slab reaches; trim 0 lists every cell of the box. For
// trim 1 (at most kLineRows rows of at most kLineNx cells) the runs are one
// byte per row in the Gaussian's line of kLineRows bytes: the first and
// last cell as offsets from x0 (low and high 4 bits), kRunEmpty for a row
// with none. For trim 2 they are nrec RowRecs, one per row with cells, in
// row order, from the Gaussian's record base.
struct alignas(16) CellBox {
    int4 lo, hi;
};
constexpr uint32_t kLineRows = 64;
constexpr uint32_t kLineNx = 16;
constexpr uint32_t kRunEmpty = 0x0Fu;
// Trimmed boxes have at most kTrimRowsMax rows of at most kRecNxMax cells
// (RowRec's 16-bit fields); larger ones keep every cell.
constexpr uint32_t kTrimRowsMax = 4096;
constexpr uint32_t kRecNxMax = 65535;
// A row with cells of a trim-2 box: the box's cells in earlier rows, the
// row, and its first cell as an offset from x0 (its length is the next
// record's pos, or the box's count, minus pos).
struct RowRec {
    uint32_t pos;
    uint16_t row, first;
};

__device__ __forceinline__ uint32_t run_first(uint32_t code) { return code & 15u; }
__device__ __forceinline__ uint32_t run_len(uint32_t code) {
    const uint32_t a = code & 15u, b = code >> 4;
    return b >= a ? b - a + 1 : 0u;
}



// Read-only views in the constant address space: loads through them with a
// wave-uniform address become scalar loads into SGPRs.
typedef float f4v __attribute__((ext_vector_type(4)));
typedef int i4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(4))) const f4v ConstF4;
typedef __attribute__((address_space(4))) const i4v ConstI4;
typedef __attribute__((address_space(4))) const uint32_t ConstU32;

__device__ __forceinline__ CellBox load_box_uniform(const CellBox *box, uint32_t g) {
    ConstI4 *p = (ConstI4 *)box + 2 * (size_t)g;
    const i4v a = p[0], b = p[1];
    CellBox c;
    c.lo = make_int4(a.x, a.y, a.z, a.w);
    c.hi = make_int4(b.x, b.y, b.z, b.w);
    return c;
}

// --- float helpers ---------------------------------------------------------

__device__ __forceinline__ float fmaf_(float a, float b, float c) { return __builtin_fmaf(a, b, c); }

// 2^x through the hardware transcendental unit (v_exp_f32). Arguments here
// are in [-6.65, 0], far from the denormal range.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// --- cross-lane helpers ------------------------------------------------------

__device__ __forceinline__ uint32_t lane_id() {
    return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over each row of 16 lanes; every lane of the row receives the total.
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_ror:4, row_ror:8.
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x124>(x);
    x += dpp_f<0x128>(x);
    return x;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

// Lane masks of comparisons (bit l: lane l active and the comparison true),
// straight from the compare instruction.
__device__ __forceinline__ uint64_t mask_le_f(float a, float b) { return __builtin_amdgcn_fcmpf(a, b, 5); }
__device__ __forceinline__ uint64_t mask_lt_u(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, 36); }
__device__ __forceinline__ uint64_t mask_le_u(uint32_t a, uint32_t b) { return __builtin_amdgcn_uicmp(a, b, 37); }

// x of lane l ^ 16, within each half of the wave (ds_swizzle, xor mask 16)
__device__ __forceinline__ float swz_xor16(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
}

// x of lane l ^ 32 (ds_bpermute; every lane must be active)
__device__ __forceinline__ float perm_xor32(float x, uint32_t lane) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((int)((lane ^ 32u) << 2), __builtin_bit_cast(int, x)));
}

__device__ __forceinline__ float readfirst_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}
__device__ __forceinline__ float readlane_f(float x, uint32_t l) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), (int)l));
}

__device__ __forceinline__ uint32_t umax_(uint32_t a, uint32_t b) { return a > b ? a : b; }

// Wave-uniform maximum of a 32-bit value (every lane must be active): DPP
// within each row of 16 lanes, then the four row results by readlane.
__device__ __forceinline__ uint32_t wave_max_uniform(uint32_t x) {
    x = umax_(x, dpp_u<0xB1>(x));
    x = umax_(x, dpp_u<0x4E>(x));
    x = umax_(x, dpp_u<0x124>(x));
    x = umax_(x, dpp_u<0x128>(x));
    return umax_(umax_(__builtin_amdgcn_readlane(x, 0), __builtin_amdgcn_readlane(x, 16)),
                 umax_(__builtin_amdgcn_readlane(x, 32), __builtin_amdgcn_readlane(x, 48)));
}

// Inclusive scan of a 32-bit value across the 64 lanes of a wave (sum or max).
// The sum runs on DPP alone and needs all 64 lanes active: row_shr 1, 2, 4,
// 8 scan each row of 16 (lanes without a source add 0), then row_bcast:15
// adds row 0's total to row 1 and row 2's to row 3, and row_bcast:31 adds the
// total of rows 0-1 to rows 2 and 3.
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t x) {
    x += dpp_u<0x111>(x);
    x += dpp_u<0x112>(x);
    x += dpp_u<0x114>(x);
    x += dpp_u<0x118>(x);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);
    return x;
}

__device__ __forceinline__ uint64_t wave_incl_sum64(uint64_t x) {
    const uint32_t lane = lane_id();
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        uint64_t y = __shfl_up(x, o, 64);
        if (lane >= (uint32_t)o) x += y;
    }
    return x;
}

__device__ __forceinline__ uint32_t wincl(uint32_t x) { return wave_incl_sum(x); }
__device__ __forceinline__ uint64_t wincl(uint64_t x) { return wave_incl_sum64(x); }

// Exclusive scan of one value per thread over the workgroup (kBlock
// threads); *total gets the
// workgroup sum. lds needs kWavesPerBlock entries.
template <typename T>
__device__ __forceinline__ T block_excl_scan(T x, T *lds, T *total) {
    const uint32_t tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    T incl = wincl(x);
    if (lane == kWave - 1) lds[wave] = incl;
    __syncthreads();
    T wpre = 0, tot = 0;
#pragma unroll
    for (uint32_t w = 0; w < (uint32_t)kWavesPerBlock; ++w) {
        T v = lds[w];
        if (w < wave) wpre += v;
        tot += v;
    }
    __syncthreads();
    *total = tot;
    return wpre + incl - x;
}

// The max scan takes the sum's DPP steps (lanes without a source see 0);
// all 64 lanes must be active.
__device__ __forceinline__ uint32_t wave_incl_max(uint32_t x) {
    x = umax_(x, dpp_u<0x111>(x));
    x = umax_(x, dpp_u<0x112>(x));
    x = umax_(x, dpp_u<0x114>(x));
    x = umax_(x, dpp_u<0x118>(x));
    x = umax_(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false));
    x = umax_(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false));
    return x;
}

// Map a linear block id so that consecutive work lands on one XCD: blocks
// are dispatched round-robin over the 8 XCDs, each with its own L2, so block
// b runs on XCD b % 8. Blocks past the last full group of 8 keep their id.
__device__ __forceinline__ uint32_t xcd_block(uint32_t b, uint32_t nblocks) {
    const uint32_t full = nblocks & ~7u;
    if (b >= full) return b;
    return (b & 7u) * (full >> 3) + (b >> 3);
}

// Blocks are dealt round-robin over the 8 XCDs (block b on XCD b % 8). In
// each window of 8 K blocks the K blocks of XCD x take K consecutive ids,
// so that neighbouring work shares that XCD's L2 while the windows still
// spread every stretch of the work over all XCDs. Blocks past the last full
// window keep their id.
template <uint32_t K>
__device__ __forceinline__ uint32_t xcd_group(uint32_t b, uint32_t nblocks) {
    const uint32_t win = 8u * K;
    const uint32_t full = nblocks - nblocks % win;
    if (b >= full) return b;
    const uint32_t r = b % win;
    return (b - r) + (r & 7u) * K + (r >> 3);
}

// --- host side ---------------------------------------------------------------

struct Stream {
    hipStream_t s;
};

// Kernel timing hooks (api.cpp): every launcher brackets its kernels.
void prof_begin(const char *name, hipStream_t s);
void prof_end(const char *name, hipStream_t s);

// Exclusive scans. Workspace: scan_work_bytes(n) bytes. out may equal in.
size_t scan_work_bytes(int64_t n, int elem_bytes);
hipError_t exclusive_scan_u32(const uint32_t *in, uint32_t *out, int64_t n, void *work, hipStream_t s);
hipError_t exclusive_scan_u64(const uint64_t *in, uint64_t *out, int64_t n, void *work, hipStream_t s);
// exclusive scan of n elements; *total receives their sum
hipError_t exclusive_scan_u64_total(const uint64_t *in, uint64_t *out, int64_t n, uint64_t *total, void *work,
                                    hipStream_t s);
// count[0..n) -> exclusive offsets in place, given group_prefix = the
// exclusive scan of the counts' sums over groups of 64 followed by their
// total; tile_first[t] (t < ntiles) = the segment holding element
// t * tile_size
hipError_t pair_offsets(uint64_t *count, int64_t n, const uint64_t *group_prefix, uint32_t *tile_first,
                        int64_t ntiles, uint32_t tile_size, hipStream_t s);

// Stable LSD radix sort of (key, value) pairs by the low `bits` key bits
// (radix.h has the tile geometry). Passes alternate between the two buffer
// pairs; radix_passes(bits) tells which one holds the result.
struct RadixLayout {
    uint32_t *table;       // [ndig][nb] tile counts, scanned in place
    uint32_t *digit_tot;   // [ndig] digit totals of the pass
    uint32_t nb;           // tiles
    int passes, dbits;
    size_t bytes;
};
struct RadixPass0 {       // lets the producer of the keys count the first digit
    uint32_t *table;       // null: the sort counts it itself
    uint32_t nb;
    uint32_t mask;
};
RadixLayout radix_layout(void *work, int64_t n, int bits);
size_t radix_work_bytes(int64_t n, int bits);
RadixPass0 radix_pass0(void *work, int64_t n, int bits);
int radix_passes(int bits);
hipError_t radix_sort_pairs(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, int64_t n, int bits, void *work,
                            hipStream_t s, bool pass0_ready);

// offsets[k] = number of sorted keys < k, k = 0..nkeys (nkeys+1 entries).
hipError_t key_offsets(const uint32_t *sorted_keys, int64_t n, uint32_t *offsets, int64_t nkeys, hipStream_t s);

hipError_t fill_u32(uint32_t *p, uint32_t v, int64_t n, hipStream_t s);
hipError_t fill_f32(float *p, float v, int64_t n, hipStream_t s);

// Index build pieces (index.hip).
struct GridParams {
    float lo[3], hi[3];
    float invc[3];   // cells / (hi - lo), float32
    int32_t cells[3];
    int64_t ncells;
};
// count[0..n] receives the pair count of every Gaussian (count[n] = 0) and
// block_sum[b] the sum over elements [64 b, 64 b + 64) of count
// cell_coarse[c] = 1 when cell c's box list may hold a Gaussian too small
// against the cells for the dense walk's cell-centre offsets (kOffsetCells);
// ceil(ncells / 4) words, cleared here first.
hipError_t launch_preprocess(const float *mean, const float *scale, const float *rot, const float *value,
                             const float *weight, int64_t n, const GridParams &g, float rci, Record *rec, CellBox *box,
                             uint8_t *lines, RowRec *rows, uint32_t *rbase, uint32_t *rtotal, int64_t rcap,
                             uint8_t *cell_coarse, uint64_t *count, uint64_t *block_sum, hipStream_t s);
// A Gaussian is coarse when the cell diagonal passes kOffsetCells times its
// largest scale: the forward's dense walk then evaluates the cells of its
// box as U (p - mu) (see offset_planes).
#ifndef GS_OFFSET_CELLS
#define GS_OFFSET_CELLS 64.0
#endif
constexpr double kOffsetCells = GS_OFFSET_CELLS;
// tile_first: ceil(npairs / kSortTile) words of scratch
hipError_t launch_emit(const uint64_t *pair_off, const CellBox *box, const uint8_t *lines, const RowRec *rows,
                       const uint32_t *rbase, int64_t n, int64_t npairs, const GridParams &g, uint32_t *tile_first,
                       uint32_t *keys, uint32_t *gids, const RadixPass0 &pass0, hipStream_t s);

// Sampling (sample.hip).
// The plan orders the queries by cell and, inside a cell, by the quarter of
// the cell along x that their position falls in: key kSub c + j for quarter
// j of cell c, kSub ncells outside the domain. Its offsets point_off (kSub
// ncells + 2 entries) give every cell's queries, [point_off[kSub c],
// point_off[kSub (c + 1)]), and every quarter's, so that a box row can
// start and end at a quarter of a cell.
constexpr uint32_t kSub = 4;

struct QueryParams {
    int kind;
    int32_t dims[3];
    int64_t n;           // number of outputs
    const uint32_t *voxel_ids;
    const float *points;
    float vsz[3];        // (hi - lo) / dims, float32
};

__device__ __forceinline__ float voxel_center(int32_t i, float lo, float vs) { return lo + ((float)i + 0.5f) * vs; }

// Position of query pid, each operation rounded in float32: the centre of
// voxel pid (GRID) or of the listed voxel (VOXELS), the position at the
// caller's offsets in the listed voxel, or in voxel pid without a list
// (JITTER), or the given point (POINTS). valid is false for a voxel id past
// the grid.
__device__ __forceinline__ void query_position(const QueryParams &q, const GridParams &g, uint32_t pid, float &px,
                                               float &py, float &pz, bool &valid) {
    valid = true;
    if (q.kind != 2) {
        // voxel queries: centred (0, 1) or at the caller's offsets (3)
        const uint32_t id = (q.kind == 0 || (q.kind == 3 && !q.voxel_ids)) ? pid : q.voxel_ids[pid];
        const uint32_t nx = (uint32_t)q.dims[0], ny = (uint32_t)q.dims[1], nz = (uint32_t)q.dims[2];
        const uint64_t nvox = (uint64_t)nx * ny * nz;
        if ((uint64_t)id >= nvox) {
            valid = false;
            px = py = pz = 0.0f;
            return;
        }
        const uint32_t x = id % nx, t = id / nx, y = t % ny, z = t / ny;
        if (q.kind != 3) {
            px = voxel_center((int32_t)x, g.lo[0], q.vsz[0]);
            py = voxel_center((int32_t)y, g.lo[1], q.vsz[1]);
            pz = voxel_center((int32_t)z, g.lo[2], q.vsz[2]);
        } else {
            const float *u = q.points + 3 * (uint64_t)pid;
            px = g.lo[0] + ((float)x + u[0]) * q.vsz[0];
            py = g.lo[1] + ((float)y + u[1]) * q.vsz[1];
            pz = g.lo[2] + ((float)z + u[2]) * q.vsz[2];
        }
    } else {
        px = q.points[3 * (uint64_t)pid];
        py = q.points[3 * (uint64_t)pid + 1];
        pz = q.points[3 * (uint64_t)pid + 2];
    }
}
// Sort key of every query (kSub cell + quarter of the cell along x, kSub
// ncells outside the domain), identity ids and
// the first sort digit's tile counts.
hipError_t launch_query_keys(const QueryParams &q, const GridParams &g, uint32_t *keys, uint32_t *ids,
                             const RadixPass0 &pass0, hipStream_t s);
hipError_t launch_sample_grid(const QueryParams &q, const GridParams &g, const Record *rec, const uint32_t *gids,
                              const uint32_t *cell_off, float T, float tau, float *out_v, float *out_i,
                              hipStream_t s);
// Work items of the ordered-query sampler (kept in the plan).
struct PointItems {
    uint32_t *item_off;   // [ncells + 2]
    uint32_t *items;      // [max_items]
    int64_t max_items;    // ncells + 1 + n / 64 + 1
    uint64_t *group_sum;  // [item_groups(ncells + 1) + 1] work items per 1024 buckets, (dense << 32) | sparse
    void *scan_work;      // scan of group_sum
};
// groups of 1024 buckets (plus the element after the last bucket)
inline int64_t item_groups(int64_t nbuckets) { return (nbuckets + 1 + 1023) / 1024; }
// The forward's results in plan order, kept in the plan for the backward:
// position (x, y, z, 0) and (Phi, I) of the k-th query in cell order.
struct PlanResults {
    float4 *pos;
    float2 *out;
};

// The forward's work items from the plan's per-quarter ranges (the query
// ordering's last step).
hipError_t launch_cell_items(int64_t nq, const GridParams &g, const uint32_t *point_off, const PointItems &it,
                             hipStream_t s);
// cell_coarse: the index's per-cell flags (launch_preprocess).
hipError_t launch_sample_points(const QueryParams &q, const GridParams &g, const Record *rec,
                                const uint8_t *cell_coarse,
                                const uint32_t *gids,
                                const uint32_t *cell_off, const uint32_t *order, const uint32_t *point_off,
                                const PointItems &it, float T, float tau, float *out_v, float *out_i,
                                const PlanResults &pr, hipStream_t s);

// Pairs the forward tests and those passing the cutoff (measurement), into
// totals[0] and totals[1] (device, 16 bytes); plan_keys and plan_pos are
// the sorted keys and the positions a forward left in the plan (unused for
// GRID queries).
hipError_t launch_count_sample_pairs(const QueryParams &q, const GridParams &g, const Record *rec,
                                     const uint32_t *gids, const uint32_t *cell_off, const uint32_t *plan_keys,
                                     const float4 *plan_pos, float T, unsigned long long *totals, hipStream_t s);

// Gaussians in spatial order: sorted by the cell key of their box's low
// corner (empty boxes last), so neighbouring work shares cached queries.
hipError_t launch_gauss_keys(const CellBox *box, int64_t n, const GridParams &g, int shift, uint32_t *keys,
                             uint32_t *ids, const RadixPass0 &pass0, hipStream_t s);

// Backward (backward.hip).
//
// The backward walks each Gaussian's queries by rows along x, each row cut
// to the x-range of the cutoff ellipsoid over the row's (y, z) extent: for
// grids a row of voxels; for ordered queries a row of cells, a run of the
// plan's order, cut to quarters of cells along x.

// Row geometry of the backward (host-computed).
struct BwdGeom {
    float T2;          // the cutoff the row bounds use: T (1 + 2^-7)
    float cw[2];       // ordered queries: y, z extent of a cell, 1 / invc
    float slack[2];    // widening of a row's y, z extent (float rounding)
    float ivsz0;       // grids: voxels per unit along x, 1 / vsz[0]
    float xslack;      // grids: widening of a row's voxel range, in voxels
    uint32_t K;        // kSub cells[0]: quarters of a row of cells
};

// Least value over the rectangle dy in [ay, by], dz in [az, bz] (offsets
// from the mean) of q2 = (U11 dy + U12 dz)^2 + (U22 dz)^2, the minimum of Q
// over x at fixed (y, z) for the record's triangular U. q2 is convex: its
// minimum is at dy = dz = 0 when the rectangle holds it, else on an edge,
// where it is a quadratic in one variable minimised at its clamped vertex.
__device__ __forceinline__ float slab_q2min(float U11, float U12, float U22, float ay, float by, float az,
                                            float bz) {
    if (ay <= 0.0f && by >= 0.0f && az <= 0.0f && bz >= 0.0f) return 0.0f;
    const float i11 = __builtin_amdgcn_rcpf(U11);
    const float iden = __builtin_amdgcn_rcpf(fmaf_(U12, U12, U22 * U22));
    auto q2 = [&](float dy, float dz) {
        const float a = fmaf_(U11, dy, U12 * dz), b = U22 * dz;
        return fmaf_(a, a, b * b);
    };
    // fixed dz: best dy = -U12 dz / U11; fixed dy: best dz = -U11 U12 dy / (U12^2 + U22^2)
    const float ya = fminf(fmaxf(-U12 * az * i11, ay), by), yb = fminf(fmaxf(-U12 * bz * i11, ay), by);
    const float za = fminf(fmaxf(-U11 * U12 * ay * iden, az), bz), zb = fminf(fmaxf(-U11 * U12 * by * iden, az), bz);
    return fminf(fminf(q2(ya, az), q2(yb, bz)), fminf(q2(ay, za), q2(by, zb)));
}

// x-range [xl, xh] of the points of the rectangle (offsets from the mean,
// as above) with Q <= T2, or false when there are none. At fixed (y, z) Q
// <= T2 holds for |x - xc| <= sqrt(T2 - q2) / U00 with the centre xc =
// mu_x - (U01 dy + U02 dz) / U00, linear in (dy, dz): the range spans the
// centre's extremes at the rectangle's corners, widened by the half-width
// at the rectangle's least q2, and by a few units of float32 rounding.
__device__ __forceinline__ bool slab_xrange(const Record &r, float ay, float by, float az, float bz, float T2,
                                            float &xl, float &xh) {
    const float q2 = slab_q2min(r.f2.x, r.f2.y, r.f2.z, ay, by, az, bz);
    if (!(q2 <= T2)) return false;
    const float iu = __builtin_amdgcn_rcpf(r.f1.x);
    const float w = __builtin_sqrtf(T2 - q2) * iu;
    const float c0 = r.f1.y * ay, c1 = r.f1.y * by, c2 = r.f1.z * az, c3 = r.f1.z * bz;
    const float hi = (fmaxf(c0, c1) + fmaxf(c2, c3)) * iu, lo = (fminf(c0, c1) + fminf(c2, c3)) * iu;
    const float m = (fabsf(r.f0.x) + fabsf(hi) + fabsf(lo) + w) * 0x1p-20f;
    xl = r.f0.x - hi - w - m;
    xh = r.f0.x - lo + w + m;
    return true;
}

// The plan entries [start, start + len) of row (cy, cz) of a box spanning
// cells lx .. lx + nx - 1 along x whose queries can lie within the cutoff
// T2 of the record (ordered queries): the row's y, z extent widened by the
// slack, cut to the x-range of slab_xrange, taken in quarters of cells. The
// plan's quarter of x is floor(kSub t), t = (x - lo) invc, in the same
// float32 operations, monotone in x, so every query the range admits is in.
__device__ __forceinline__ uint32_t plan_row(const Record &r, uint32_t lx, uint32_t nx, uint32_t cy, uint32_t cz,
                                             const GridParams &g, const BwdGeom &bg,
                                             const uint32_t *__restrict__ point_off, uint32_t &start) {
    start = 0;
    const float y0 = g.lo[1] + (float)cy * bg.cw[0] - bg.slack[0];
    const float y1 = g.lo[1] + (float)(cy + 1u) * bg.cw[0] + bg.slack[0];
    const float z0 = g.lo[2] + (float)cz * bg.cw[1] - bg.slack[1];
    const float z1 = g.lo[2] + (float)(cz + 1u) * bg.cw[1] + bg.slack[1];
    float xl, xh;
    if (!slab_xrange(r, y0 - r.f0.y, y1 - r.f0.y, z0 - r.f0.z, z1 - r.f0.z, bg.T2, xl, xh)) return 0;
    const float qmin = (float)(kSub * lx), qmax = (float)(kSub * (lx + nx)) - 1.0f;
    const float ql = fminf(fmaxf(floorf((float)kSub * ((xl - g.lo[0]) * g.invc[0])), qmin), qmax);
    const float qh = fminf(fmaxf(floorf((float)kSub * ((xh - g.lo[0]) * g.invc[0])), qmin), qmax);
    // the row's quarters are entries base .. base + K of the plan's offsets,
    // the last one the start of the next row of cells
    const uint32_t base = (cz * (uint32_t)g.cells[1] + cy) * bg.K;
    start = point_off[base + (uint32_t)ql];
    return point_off[base + (uint32_t)qh + 1u] - start;
}

struct BackwardBuffers {
    float *moments;        // [n_gauss][12]
    float2 *ab;            // [n] (alpha, beta) per query: plan order (ordered queries) or voxel order (grid)
    float2 *cot;           // [n] (dL/dPhi, dL/dI) packed in query order (ordered queries)
};
// Pairs the backward tests (measurement), into *total (device, 8 bytes);
// point_off: the plan's offsets (ordered queries).
hipError_t launch_count_backward_pairs(const QueryParams &q, const GridParams &g, const BwdGeom &bg,
                                      const Record *rec, const CellBox *box, int64_t n_gauss,
                                      const uint32_t *point_off, unsigned long long *total, hipStream_t s);
// n_pairs: the index's pair count (it sets how many Gaussians share a wave)
hipError_t launch_backward(const QueryParams &q, const GridParams &g, const BwdGeom &bg, const Record *rec,
                           const CellBox *box, const uint32_t *gorder, int64_t n_gauss, int64_t n_pairs,
                           const uint32_t *order, const uint32_t *point_off, const float4 *plan_pos,
                           const float2 *plan_out, const float *value, const float *influence,
                           const float *grad_value, const float *grad_influence, float T,
                           const BackwardBuffers &b, const float *scale, const float *rot, float *d_mean,
                           float *d_scale, float *d_rot, float *d_value, float *d_weight, hipStream_t s);

// Densification (densify.hip).
size_t densify_work_bytes(int64_t n_in, int64_t nq);

// Training epilogue (train.hip). cap <= 0 disables the soft cap.
size_t loss_work_bytes(int64_t n);
hipError_t launch_activate(int64_t n, const float *log_scale, const float *value_logit, const float *weight_logit,
                           double cap, float *scale, float *value, float *weight, hipStream_t s);
hipError_t launch_activate_backward(int64_t n, const float *log_scale, const float *value_logit,
                                    const float *weight_logit, double cap, const float *d_scale,
                                    const float *d_value, const float *d_weight, float *d_log_scale,
                                    float *d_value_logit, float *d_weight_logit, hipStream_t s);

}  // namespace gs
