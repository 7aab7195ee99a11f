// C-ABI of the library (include/gs.h): argument validation, workspace
// layout, the three entry points, and kernel timing.
#include "../../include/gs.h"
#include "../../include/gs_train.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"
#include "radix.h"

namespace gs {
hipError_t launch_loss(int64_t n, const float *value, const float *influence, const float *target,
                       const uint8_t *defined, float tau, float eps, float lambda_fn, float lambda_fp,
                       float *grad_value, float *grad_influence, gs_loss_terms *terms, void *work, hipStream_t s);
hipError_t launch_sample_gauss_major(const QueryParams &q, const GridParams &g, const BwdGeom &bg, const Record *rec,
                                     const CellBox *box, const uint32_t *gorder,
                                     int64_t n_gauss, const uint32_t *order, const uint32_t *point_off, float T,
                                     float tau, float *out_v, float *out_i, const PlanResults &pr, void *work,
                                     hipStream_t s);
size_t gauss_major_work_bytes(int64_t nq);
hipError_t launch_densify(const gs_params &in, int64_t n_in, const float *weight, float tau2, const QueryParams &q,
                          const GridParams &g, const float *value, const float *influence, const float *target,
                          const uint8_t *defined, float tau, float new_log_scale, float new_weight_logit,
                          int64_t max_new, int64_t capacity, const gs_params &out, int32_t *source, void *work,
                          long long **n_out_dev, hipStream_t s);
}

using namespace gs;

namespace {

thread_local std::string g_err;

gs_status fail(gs_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
gs_status fail(gs_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

gs_status hip_fail(hipError_t e, const char *what) {
    return fail(GS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define GS_TRY(expr, what)                                   \
    do {                                                     \
        hipError_t e_ = (expr);                              \
        if (e_ != hipSuccess) return hip_fail(e_, (what));   \
    } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Bump allocator over a caller workspace (computes the layout when base is null).
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base((char *)b) {}
    template <typename T>
    T *take(size_t count) {
        T *p = base ? (T *)(base + off) : nullptr;
        off = align_up(off + count * sizeof(T));
        return p;
    }
};

int bits_for(int64_t nkeys) {  // bits needed to hold keys 0..nkeys-1
    int b = 0;
    while (b < 40 && ((int64_t)1 << b) < nkeys) ++b;
    return b;
}

bool grid_valid(const gs_grid *g, std::string *why) {
    if (!g) {
        *why = "grid is null";
        return false;
    }
    int64_t nc = 1;
    for (int j = 0; j < 3; ++j) {
        if (!(std::isfinite(g->lo[j]) && std::isfinite(g->hi[j]) && g->hi[j] > g->lo[j])) {
            *why = "grid box must be finite with hi > lo on every axis";
            return false;
        }
        if (g->cells[j] <= 0) {
            *why = "grid cells must be positive";
            return false;
        }
        nc *= g->cells[j];
        if (nc >= ((int64_t)1 << 31)) {
            *why = "grid has 2^31 cells or more";
            return false;
        }
    }
    return true;
}

int64_t ncells_of(const gs_grid *g) { return (int64_t)g->cells[0] * g->cells[1] * g->cells[2]; }

GridParams grid_params(const gs_grid *g) {
    GridParams p;
    for (int j = 0; j < 3; ++j) {
        p.lo[j] = g->lo[j];
        p.hi[j] = g->hi[j];
        volatile float ext = g->hi[j] - g->lo[j];
        p.invc[j] = (float)g->cells[j] / ext;
        p.cells[j] = g->cells[j];
    }
    p.ncells = ncells_of(g);
    return p;
}

// Gaussians are ordered by the cell key of their box corner, coarsened to
// at most 10 bits so that one radix pass sorts them.
int gauss_order_full_bits(const gs_grid *g) { return bits_for(ncells_of(g) + 1); }
int gauss_order_shift(const gs_grid *g) {
    const int b = gauss_order_full_bits(g);
    return b > 10 ? b - 10 : 0;
}
int gauss_order_bits(const gs_grid *g) { return gauss_order_full_bits(g) - gauss_order_shift(g); }

// Index workspace layout.
struct IndexWork {
    CellBox *box;        // [n] cell boxes (first: the tests read them back)
    Record *rec;         // [n] evaluation records
    uint8_t *lines;      // [n][kLineRows] row-run bytes of the trim-1 boxes
    uint8_t *cell_coarse;  // [ncells, 4-byte words] cells holding a Gaussian too small for the offsets
    uint32_t *rbase;     // [n] first row record of each trim-2 box
    uint32_t *rtotal;    // row records taken so far (one word)
    uint32_t *gorder;    // [n] Gaussians in spatial order
    uint32_t *gkeys;     // [n] their sort keys
    uint32_t *gsort_k;   // [n] sort scratch
    uint32_t *gsort_v;   // [n] sort scratch
    void *gsort_work;
    uint64_t *pair_off;  // [n + 1]
    uint64_t *pair_sum;  // [ceil((n + 1) / 64)] pair counts per 64 Gaussians, then their scan
    void *scan_work;
    uint32_t *tile_first;  // [pair tiles] first Gaussian of every emit tile
    uint32_t *keys_alt;
    uint32_t *gids_alt;
    RowRec *rows;        // [capacity] row records of the trim-2 boxes (each row has a pair)
    void *radix_work;
    size_t bytes;
};

// pair counts are summed per 64 Gaussians (the preprocess workgroups, the
// last one holding count[n] = 0); the scan of the sums of the first
// ceil(n / 64) groups is followed by their total
int64_t pair_groups_scanned(int64_t n) { return (n + 63) / 64; }
int64_t tile_first_len(int64_t capacity) { return ((capacity > 0 ? capacity : 1) + kSortTile - 1) / kSortTile + 1; }

IndexWork index_layout(void *base, int64_t n, const gs_grid *g, int64_t capacity) {
    Carver c(base);
    IndexWork w;
    const size_t n1 = (size_t)(n > 0 ? n : 1);
    w.box = c.take<CellBox>(n1);
    w.rec = c.take<Record>(n1);
    w.lines = c.take<uint8_t>(n1 * kLineRows);
    w.cell_coarse = c.take<uint8_t>((size_t)((ncells_of(g) + 3) / 4) * 4);
    w.rbase = c.take<uint32_t>(n1);
    w.rtotal = c.take<uint32_t>(4);
    w.gorder = c.take<uint32_t>(n1);
    w.gkeys = c.take<uint32_t>(n1);
    w.gsort_k = c.take<uint32_t>(n1);
    w.gsort_v = c.take<uint32_t>(n1);
    w.gsort_work = c.take<char>(radix_work_bytes((int64_t)n1, gauss_order_bits(g)));
    w.pair_off = c.take<uint64_t>((size_t)n + 1);
    w.pair_sum = c.take<uint64_t>((size_t)pair_groups_scanned(n) + 1);
    w.scan_work = c.take<char>(scan_work_bytes(pair_groups_scanned(n), 8));
    w.tile_first = c.take<uint32_t>((size_t)tile_first_len(capacity));
    const int64_t cap = capacity > 0 ? capacity : 1;
    w.keys_alt = c.take<uint32_t>((size_t)cap);
    w.gids_alt = c.take<uint32_t>((size_t)cap);
    w.rows = c.take<RowRec>((size_t)cap);
    w.radix_work = c.take<char>(radix_work_bytes(cap, bits_for(ncells_of(g))));
    w.bytes = c.off;
    return w;
}

// Plan layout (VOXELS and POINTS queries).
struct Plan {
    uint32_t *keys;      // [n] sorted cell keys (ncells = outside)
    uint32_t *order;     // [n] query ids in cell order
    uint32_t *keys_alt;  // [n]
    uint32_t *order_alt; // [n]
    uint32_t *point_off; // [kSub ncells + 2]
    void *radix_work;
    PointItems items;
    PlanResults res;
    size_t bytes;
};

Plan plan_layout(void *base, int64_t n, int64_t ncells) {
    Carver c(base);
    Plan p;
    const size_t m = (size_t)(n > 0 ? n : 1);
    p.keys = c.take<uint32_t>(m);
    p.order = c.take<uint32_t>(m);
    p.keys_alt = c.take<uint32_t>(m);
    p.order_alt = c.take<uint32_t>(m);
    p.point_off = c.take<uint32_t>((size_t)kSub * ncells + 2);
    p.radix_work = c.take<char>(radix_work_bytes(n > 0 ? n : 1, bits_for((int64_t)kSub * ncells + 1)));
    p.items.item_off = c.take<uint32_t>((size_t)ncells + 2);
    p.items.max_items = ncells + 1 + (n > 0 ? n : 0) / 64 + 1;
    p.items.items = c.take<uint32_t>((size_t)p.items.max_items);
    p.items.group_sum = c.take<uint64_t>((size_t)item_groups(ncells + 1) + 1);
    p.items.scan_work = c.take<char>(scan_work_bytes(item_groups(ncells + 1), 8));
    // 64 spare entries: the backward's lanes past a Gaussian's last point
    // read up to 63 entries beyond the last row of the plan
    p.res.pos = c.take<float4>(m + kWave);
    p.res.out = c.take<float2>(m);
    p.bytes = c.off;
    return p;
}

bool query_valid(const gs_query *q, std::string *why) {
    if (!q) {
        *why = "query is null";
        return false;
    }
    int64_t nv = 1;
    if (q->kind == GS_QUERY_GRID || q->kind == GS_QUERY_VOXELS || q->kind == GS_QUERY_JITTER) {
        for (int j = 0; j < 3; ++j) {
            if (q->dims[j] <= 0) {
                *why = "query dims must be positive";
                return false;
            }
            nv *= q->dims[j];
        }
        if (nv >= ((int64_t)1 << 32)) {
            *why = "query grid has 2^32 voxels or more";
            return false;
        }
    }
    if (q->kind == GS_QUERY_GRID) return true;
    if (q->kind != GS_QUERY_VOXELS && q->kind != GS_QUERY_POINTS && q->kind != GS_QUERY_JITTER) {
        *why = "unknown query kind";
        return false;
    }
    if (q->n < 0 || q->n >= ((int64_t)1 << 31)) {
        *why = "query count must be in [0, 2^31)";
        return false;
    }
    if (q->n > 0 && q->kind == GS_QUERY_VOXELS && !q->voxel_ids) {
        *why = "voxel_ids is null";
        return false;
    }
    if (q->n > 0 && q->kind == GS_QUERY_POINTS && !q->points) {
        *why = "points is null";
        return false;
    }
    if (q->n > 0 && q->kind == GS_QUERY_JITTER && !q->points) {
        *why = "jitter offsets (points) are null";
        return false;
    }
    if (q->kind == GS_QUERY_JITTER && !q->voxel_ids && q->n != nv) {
        *why = "a jitter query without voxel_ids covers every voxel: n must equal the voxel count";
        return false;
    }
    return true;
}

int64_t query_count(const gs_query *q) {
    if (q->kind == GS_QUERY_GRID) return (int64_t)q->dims[0] * q->dims[1] * q->dims[2];
    return q->n;
}

QueryParams query_params(const gs_query *q, const gs_grid *g) {
    QueryParams p;
    p.kind = q->kind;
    for (int j = 0; j < 3; ++j) p.dims[j] = q->kind == GS_QUERY_POINTS ? 1 : q->dims[j];
    p.n = query_count(q);
    p.voxel_ids = q->voxel_ids;
    p.points = q->points;
    for (int j = 0; j < 3; ++j) {
        volatile float ext = g->hi[j] - g->lo[j];
        p.vsz[j] = ext / (float)p.dims[j];
    }
    return p;
}

bool gauss_valid(const gs_gaussians *g, std::string *why) {
    if (!g) {
        *why = "gaussians is null";
        return false;
    }
    if (g->n < 0 || g->n >= ((int64_t)1 << 31)) {
        *why = "number of Gaussians must be in [0, 2^31)";
        return false;
    }
    if (g->n > 0 && (!g->mean || !g->scale || !g->rot || !g->value || !g->weight)) {
        *why = "a Gaussian parameter array is null";
        return false;
    }
    return true;
}

bool aligned(const void *p) { return ((uintptr_t)p % kAlign) == 0; }

// The cutoff on the records' Q' = Q log2(e) / 2: G >= tau reads Q' <= log2(1/tau).
float cutoff_T(float tau) { return (float)std::log2(1.0 / (double)tau); }
float index_radius(float tau) {
    const double rc = std::sqrt(2.0 * std::log(1.0 / (double)tau));
    return (float)(rc * (1.0 + 1.0 / 1024.0));
}

// The backward's row geometry for a grid and query (see BwdGeom).
BwdGeom bwd_geom(const GridParams &gp, const QueryParams &qp, float T) {
    BwdGeom b;
    b.T2 = (float)((double)T * (1.0 + 1.0 / 128.0));
    for (int j = 0; j < 2; ++j) {
        b.cw[j] = (float)(1.0 / (double)gp.invc[j + 1]);
        b.slack[j] = (float)(std::ldexp(1.0, -18) * (std::fabs((double)gp.lo[j + 1]) + std::fabs((double)gp.hi[j + 1])));
    }
    const double ext0 = (double)gp.hi[0] - (double)gp.lo[0];
    b.ivsz0 = qp.kind == GS_QUERY_GRID ? (float)(1.0 / (double)qp.vsz[0]) : 0.0f;
    b.xslack = qp.kind == GS_QUERY_GRID
                   ? (float)(std::ldexp(1.0, -20) * (double)qp.dims[0] *
                                 (1.0 + (std::fabs((double)gp.lo[0]) + std::fabs((double)gp.hi[0])) / ext0) +
                             std::ldexp(1.0, -12))
                   : 0.0f;
    b.K = (uint32_t)(kSub * gp.cells[0]);
    return b;
}

// Backward workspace layout.
struct BwdWork {
    BackwardBuffers b;
    size_t bytes;
};

BwdWork bwd_layout(void *base, const gs_index *index, const gs_query *q) {
    Carver c(base);
    BwdWork w;
    const int64_t n = index->n_gauss;
    const int64_t nq = query_count(q);
    const size_t mq = (size_t)(nq > 0 ? nq : 1);
    w.b.moments = c.take<float>((size_t)(n > 0 ? n : 1) * 12);
    w.b.ab = c.take<float2>(mq);
    w.b.cot = q->kind != GS_QUERY_GRID ? c.take<float2>(mq) : nullptr;
    w.bytes = c.off;
    return w;
}

// ---------------------------------------------------------------------------
// Kernel timing.

struct ProfRec {
    const char *name;
    hipEvent_t a, b;
};
struct ProfAgg {
    const char *name;
    int64_t count;
    double ms;
};
bool g_prof_on = false;
std::string g_prof_only;             // record only this kernel when non-empty
std::vector<ProfRec> g_prof_open;   // begun, not yet ended
std::vector<ProfRec> g_prof_done;   // ended, not yet read
std::vector<hipEvent_t> g_prof_pool;
std::vector<ProfAgg> g_prof_agg;

hipEvent_t prof_event() {
    if (!g_prof_pool.empty()) {
        hipEvent_t e = g_prof_pool.back();
        g_prof_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

void prof_collect() {
    for (const ProfRec &r : g_prof_done) {
        float ms = 0.0f;
        if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
            bool found = false;
            for (ProfAgg &a : g_prof_agg)
                if (std::strcmp(a.name, r.name) == 0) {
                    a.count++;
                    a.ms += ms;
                    found = true;
                    break;
                }
            if (!found) g_prof_agg.push_back({r.name, 1, (double)ms});
        }
        g_prof_pool.push_back(r.a);
        g_prof_pool.push_back(r.b);
    }
    g_prof_done.clear();
}

// A pinned host word per host thread for the pair count read back by the
// index build, with the event that marks its copy (created on first use,
// kept until the process ends).
struct PinnedCount {
    uint64_t *value = nullptr;
    hipEvent_t copied = nullptr;
};

PinnedCount *pinned_count() {
    static thread_local PinnedCount pc;
    if (!pc.value) {
        void *p = nullptr;
        if (hipHostMalloc(&p, sizeof(uint64_t), hipHostMallocDefault) != hipSuccess) return nullptr;
        if (hipEventCreateWithFlags(&pc.copied, hipEventDisableTiming) != hipSuccess) {
            (void)hipHostFree(p);
            return nullptr;
        }
        pc.value = (uint64_t *)p;
    }
    return &pc;
}

// The query ordering both forwards share (Sec. 5.1.1's point index in the
// form of a cell ordering): cell key per query, stable radix sort, per-cell
// ranges. Leaves the order and ranges in the plan.
gs_status order_queries(const char *who, const QueryParams &qp, const GridParams &gp, int64_t nq, void *plan,
                        size_t plan_bytes, Plan *out, hipStream_t stream) {
    const size_t need = plan_layout(nullptr, nq, gp.ncells).bytes;
    if (!plan || plan_bytes < need || !aligned(plan))
        return fail(GS_ERR_WORKSPACE, "%s: plan needs %zu bytes, 256-byte aligned (got %zu)", who, need, plan_bytes);
    Plan p = plan_layout(plan, nq, gp.ncells);
    const int bits = bits_for((int64_t)kSub * gp.ncells + 1);
    const bool odd = (radix_passes(bits) & 1) != 0;
    uint32_t *ek = odd ? p.keys_alt : p.keys, *ev = odd ? p.order_alt : p.order;
    uint32_t *ak = odd ? p.keys : p.keys_alt, *av = odd ? p.order : p.order_alt;
    GS_TRY(launch_query_keys(qp, gp, ek, ev, radix_pass0(p.radix_work, nq, bits), stream), "query keys");
    GS_TRY(radix_sort_pairs(ek, ev, ak, av, nq, bits, p.radix_work, stream, true), "query sort");
    GS_TRY(key_offsets(p.keys, nq, p.point_off, (int64_t)kSub * gp.ncells + 1, stream), "query ranges");
    *out = p;
    return GS_OK;
}

}  // namespace

namespace gs {

void prof_begin(const char *name, hipStream_t s) {
    if (!g_prof_on) return;
    if (!g_prof_only.empty() && g_prof_only != name) return;
    hipEvent_t a = prof_event();
    if (!a) return;
    (void)hipEventRecord(a, s);
    g_prof_open.push_back({name, a, nullptr});
}

void prof_end(const char *name, hipStream_t s) {
    if (!g_prof_on) return;
    for (size_t i = g_prof_open.size(); i-- > 0;) {
        if (g_prof_open[i].name == name || std::strcmp(g_prof_open[i].name, name) == 0) {
            ProfRec r = g_prof_open[i];
            g_prof_open.erase(g_prof_open.begin() + (long)i);
            r.b = prof_event();
            if (!r.b) {
                g_prof_pool.push_back(r.a);
                return;
            }
            (void)hipEventRecord(r.b, s);
            g_prof_done.push_back(r);
            if (g_prof_done.size() > 4096) prof_collect();
            return;
        }
    }
}

}  // namespace gs

// Workspace of gs_sample_backward_noalloc: a file-scope device array, one
// copy per GPU, held until the process ends. Host code never uses the
// array's name as an address: each device's copy is located once with
// hipGetSymbolAddress (that device current) and the address kept per device.
namespace {

constexpr size_t kNoAllocScratchBytes = GS_BACKWARD_NOALLOC_MAX_BYTES;
__device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's copy of scratch, or null with *err set.
void *scratch_address(hipError_t *err) {
    int dev = 0;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess) return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        *err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (*err != hipSuccess) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

const char *gs_last_error(void) { return g_err.c_str(); }

int gs_version(void) { return 100; }

void gs_profile_enable(int on) { g_prof_on = on != 0; }

void gs_profile_select(const char *name) { g_prof_only = name ? name : ""; }

void gs_profile_reset(void) {
    prof_collect();
    g_prof_agg.clear();
}

int gs_profile_read(const char **names, int64_t *counts, double *total_ms, int max_entries) {
    prof_collect();
    const int n = (int)g_prof_agg.size();
    for (int i = 0; i < n && i < max_entries; ++i) {
        if (names) names[i] = g_prof_agg[i].name;
        if (counts) counts[i] = g_prof_agg[i].count;
        if (total_ms) total_ms[i] = g_prof_agg[i].ms;
    }
    return n;
}

int64_t gs_query_size(const gs_query *query) {
    std::string why;
    if (!query_valid(query, &why)) return -1;
    return query_count(query);
}

size_t gs_index_work_bytes(int64_t n_gauss, const gs_grid *grid, int64_t capacity) {
    std::string why;
    if (n_gauss < 0 || capacity < 0 || !grid_valid(grid, &why)) return (size_t)-1;
    return index_layout(nullptr, n_gauss, grid, capacity).bytes;
}

gs_status gs_build_index(const gs_gaussians *gauss, const gs_grid *grid, float tau, gs_index *index,
                         hipStream_t stream) {
    std::string why;
    if (!gauss_valid(gauss, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: %s", why.c_str());
    if (!grid_valid(grid, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: %s", why.c_str());
    if (!(tau > 0.0f && tau < 1.0f)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: tau must be in (0, 1)");
    if (!index) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: index is null");
    if (index->capacity < 0) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: negative capacity");
    if (!index->cell_offsets) return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: cell_offsets is null");
    if (index->capacity > 0 && (!index->keys || !index->gids))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_build_index: keys/gids are null");
    const int64_t n = gauss->n;
    const size_t need = index_layout(nullptr, n, grid, index->capacity).bytes;
    if (!index->work || index->work_bytes < need || !aligned(index->work))
        return fail(GS_ERR_WORKSPACE, "gs_build_index: workspace needs %zu bytes, 256-byte aligned (got %zu)", need,
                    index->work_bytes);
    index->n_pairs = -1;
    index->n_gauss = n;
    index->grid = *grid;
    index->tau = tau;
    const GridParams gp = grid_params(grid);
    const int64_t ncells = gp.ncells;
    IndexWork w = index_layout(index->work, n, grid, index->capacity);

    GS_TRY(launch_preprocess(gauss->mean, gauss->scale, gauss->rot, gauss->value, gauss->weight, n, gp,
                             index_radius(tau), w.rec, w.box, w.lines, w.rows, w.rbase, w.rtotal, index->capacity,
                             w.cell_coarse, w.pair_off, w.pair_sum, stream),
           "gs_build_index: preprocess");
    {
        // groups past ceil(n / 64) hold only count[n] = 0: their prefix is the total
        const int64_t G = pair_groups_scanned(n);
        if (G > 0)
            GS_TRY(exclusive_scan_u64_total(w.pair_sum, w.pair_sum, G, w.pair_sum + G, w.scan_work, stream),
                   "gs_build_index: scan of the group sums");
        else
            GS_TRY(fill_u32((uint32_t *)w.pair_sum, 0u, 2, stream), "gs_build_index: scan of the group sums");
    }
    GS_TRY(pair_offsets(w.pair_off, n + 1, w.pair_sum, w.tile_first, tile_first_len(index->capacity), kSortTile, stream),
           "gs_build_index: pair offsets");
    // the pair count goes to a pinned host word; the host waits for that copy
    // only, while the device goes on with the Gaussian sort
    PinnedCount *pc = pinned_count();
    if (!pc) return fail(GS_ERR_HIP, "gs_build_index: cannot set up the pinned pair-count slot");
    GS_TRY(hipMemcpyAsync(pc->value, w.pair_off + n, sizeof(uint64_t), hipMemcpyDeviceToHost, stream),
           "gs_build_index: reading the pair count");
    GS_TRY(hipEventRecord(pc->copied, stream), "gs_build_index: reading the pair count");
    // the Gaussians' visiting order needs only the boxes: the device sorts
    // them while the host waits for the pair count
    {
        // spatial visiting order of the Gaussians (sorted by box corner cell)
        const int gbits = gauss_order_bits(grid);
        const bool godd = (radix_passes(gbits) & 1) != 0;
        uint32_t *k0 = godd ? w.gsort_k : w.gkeys, *v0 = godd ? w.gsort_v : w.gorder;
        uint32_t *k1 = godd ? w.gkeys : w.gsort_k, *v1 = godd ? w.gorder : w.gsort_v;
        GS_TRY(launch_gauss_keys(w.box, n, gp, gauss_order_shift(grid), k0, v0, radix_pass0(w.gsort_work, n, gbits),
                                 stream),
               "gs_build_index: Gaussian keys");
        GS_TRY(radix_sort_pairs(k0, v0, k1, v1, n, gbits, w.gsort_work, stream, true),
               "gs_build_index: Gaussian order");
    }
    GS_TRY(hipEventSynchronize(pc->copied), "gs_build_index: waiting for the pair count");
    const uint64_t P = *pc->value;
    index->n_pairs = (int64_t)P;
    if ((int64_t)P > index->capacity || P >= ((uint64_t)1 << 32))
        return fail(GS_ERR_CAPACITY, "gs_build_index: %llu pairs exceed the capacity %lld",
                    (unsigned long long)P, (long long)index->capacity);
    if (P == 0) {
        GS_TRY(fill_u32(index->cell_offsets, 0u, ncells + 1, stream), "gs_build_index: offsets");
        return GS_OK;
    }
    const int bits = bits_for(ncells);
    const bool odd = (radix_passes(bits) & 1) != 0;
    // emit where the sort's last pass lands in keys/gids
    uint32_t *ek = odd ? w.keys_alt : index->keys, *ev = odd ? w.gids_alt : index->gids;
    uint32_t *ak = odd ? index->keys : w.keys_alt, *av = odd ? index->gids : w.gids_alt;
    GS_TRY(launch_emit(w.pair_off, w.box, w.lines, w.rows, w.rbase, n, (int64_t)P, gp, w.tile_first, ek, ev,
                       radix_pass0(w.radix_work, (int64_t)P, bits), stream),
           "gs_build_index: emit");
    GS_TRY(radix_sort_pairs(ek, ev, ak, av, (int64_t)P, bits, w.radix_work, stream, true), "gs_build_index: sort");
    GS_TRY(key_offsets(index->keys, (int64_t)P, index->cell_offsets, ncells, stream), "gs_build_index: ranges");
    return GS_OK;
}

// Ordered queries (VOXELS, POINTS, JITTER) sort 32-bit keys kSub cell +
// quarter, with kSub ncells for the outside bucket: the grid must keep
// kSub ncells + 1 below 2^32.
bool ordered_grid_ok(const gs_grid *g) { return (int64_t)kSub * ncells_of(g) + 1 < ((int64_t)1 << 32); }

size_t gs_plan_bytes(const gs_query *query, const gs_grid *grid) {
    std::string why;
    if (!query_valid(query, &why) || !grid_valid(grid, &why)) return (size_t)-1;
    if (query->kind == GS_QUERY_GRID) return 0;
    if (!ordered_grid_ok(grid)) return (size_t)-1;
    return plan_layout(nullptr, query->n, ncells_of(grid)).bytes;
}

static gs_status check_index(const char *fn, const gs_gaussians *gauss, const gs_index *index) {
    std::string why;
    if (!gauss_valid(gauss, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "%s: %s", fn, why.c_str());
    if (!index) return fail(GS_ERR_INVALID_ARGUMENT, "%s: index is null", fn);
    if (index->n_pairs < 0 || index->n_pairs > index->capacity)
        return fail(GS_ERR_INVALID_ARGUMENT, "%s: the index has not been built", fn);
    if (index->n_gauss != gauss->n)
        return fail(GS_ERR_INVALID_ARGUMENT, "%s: the index was built for %lld Gaussians, not %lld", fn,
                    (long long)index->n_gauss, (long long)gauss->n);
    if (!grid_valid(&index->grid, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "%s: %s", fn, why.c_str());
    if (!index->work || !index->cell_offsets || (index->n_pairs > 0 && !index->gids))
        return fail(GS_ERR_INVALID_ARGUMENT, "%s: index buffers are null", fn);
    return GS_OK;
}

static gs_status check_query_grid(const char *fn, const gs_grid *grid, const gs_query *query) {
    std::string why;
    if (!query_valid(query, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "%s: %s", fn, why.c_str());
    if (query->kind == GS_QUERY_GRID)
        for (int j = 0; j < 3; ++j)
            if (query->dims[j] % grid->cells[j] != 0)
                return fail(GS_ERR_INVALID_ARGUMENT,
                            "%s: grid query dims must be a multiple of the index cells on every axis", fn);
    if (query->kind != GS_QUERY_GRID && !ordered_grid_ok(grid))
        return fail(GS_ERR_INVALID_ARGUMENT,
                    "%s: voxel, point and jitter queries need an index grid of fewer than 2^30 cells", fn);
    return GS_OK;
}

static gs_status check_query(const char *fn, const gs_index *index, const gs_query *query) {
    return check_query_grid(fn, &index->grid, query);
}

// The query ordering and the forward's work items (ordered queries).
static gs_status plan_queries(const char *who, const QueryParams &qp, const GridParams &gp, int64_t nq, void *plan,
                              size_t plan_bytes, Plan *out, hipStream_t stream) {
    gs_status st = order_queries(who, qp, gp, nq, plan, plan_bytes, out, stream);
    if (st != GS_OK) return st;
    GS_TRY(launch_cell_items(nq, gp, out->point_off, out->items, stream), "work items");
    return GS_OK;
}

// The point sampler over a plan that plan_queries filled.
static gs_status sample_ordered(const char *who, const gs_index *index, const QueryParams &qp, const GridParams &gp,
                                const Plan &p, float *out_value, float *out_influence, hipStream_t stream) {
    IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
    GS_TRY(launch_sample_points(qp, gp, w.rec, w.cell_coarse, index->gids, index->cell_offsets, p.order, p.point_off, p.items,
                                cutoff_T(index->tau), index->tau, out_value, out_influence, p.res, stream),
           who);
    return GS_OK;
}

gs_status gs_sample(const gs_gaussians *gauss, const gs_index *index, const gs_query *query, float *out_value,
                    float *out_influence, void *plan, size_t plan_bytes, hipStream_t stream) {
    gs_status st = check_index("gs_sample", gauss, index);
    if (st != GS_OK) return st;
    if ((st = check_query("gs_sample", index, query)) != GS_OK) return st;
    const int64_t nq = query_count(query);
    if (nq > 0 && (!out_value || !out_influence))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample: output arrays are null");
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
    const float T = cutoff_T(index->tau);
    if (query->kind == GS_QUERY_GRID) {
        GS_TRY(launch_sample_grid(qp, gp, w.rec, index->gids, index->cell_offsets, T, index->tau, out_value,
                                  out_influence, stream),
               "gs_sample: grid sampler");
        return GS_OK;
    }
    Plan p;
    if ((st = plan_queries("gs_sample", qp, gp, nq, plan, plan_bytes, &p, stream)) != GS_OK) return st;
    return sample_ordered("gs_sample: point sampler", index, qp, gp, p, out_value, out_influence, stream);
}

gs_status gs_plan_queries(const gs_query *query, const gs_grid *grid, void *plan, size_t plan_bytes,
                          hipStream_t stream) {
    std::string why;
    if (!grid_valid(grid, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_plan_queries: %s", why.c_str());
    gs_status st = check_query_grid("gs_plan_queries", grid, query);
    if (st != GS_OK) return st;
    if (query->kind == GS_QUERY_GRID) return GS_OK;
    const GridParams gp = grid_params(grid);
    const QueryParams qp = query_params(query, grid);
    Plan p;
    return plan_queries("gs_plan_queries", qp, gp, query_count(query), plan, plan_bytes, &p, stream);
}

gs_status gs_sample_planned(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                            float *out_value, float *out_influence, void *plan, size_t plan_bytes,
                            hipStream_t stream) {
    gs_status st = check_index("gs_sample_planned", gauss, index);
    if (st != GS_OK) return st;
    if ((st = check_query("gs_sample_planned", index, query)) != GS_OK) return st;
    const int64_t nq = query_count(query);
    if (nq > 0 && (!out_value || !out_influence))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_planned: output arrays are null");
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    if (query->kind == GS_QUERY_GRID) {
        IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
        GS_TRY(launch_sample_grid(qp, gp, w.rec, index->gids, index->cell_offsets, cutoff_T(index->tau), index->tau,
                                  out_value, out_influence, stream),
               "gs_sample_planned: grid sampler");
        return GS_OK;
    }
    const size_t need = plan_layout(nullptr, nq, gp.ncells).bytes;
    if (!plan || plan_bytes < need || !aligned(plan))
        return fail(GS_ERR_WORKSPACE, "gs_sample_planned: plan needs %zu bytes, 256-byte aligned (got %zu)", need,
                    plan_bytes);
    const Plan p = plan_layout(plan, nq, gp.ncells);
    return sample_ordered("gs_sample_planned: point sampler", index, qp, gp, p, out_value, out_influence, stream);
}

size_t gs_sample_gaussian_major_work_bytes(const gs_query *query) {
    std::string why;
    if (!query_valid(query, &why) || query->kind == GS_QUERY_GRID) return (size_t)-1;
    return gauss_major_work_bytes(query_count(query));
}

gs_status gs_sample_gaussian_major(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                                   float *out_value, float *out_influence, void *plan, size_t plan_bytes, void *work,
                                   size_t work_bytes, hipStream_t stream) {
    gs_status st = check_index("gs_sample_gaussian_major", gauss, index);
    if (st != GS_OK) return st;
    if ((st = check_query("gs_sample_gaussian_major", index, query)) != GS_OK) return st;
    if (query->kind == GS_QUERY_GRID)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_gaussian_major: grid queries are not supported (use gs_sample)");
    const int64_t nq = query_count(query);
    if (nq > 0 && (!out_value || !out_influence))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_gaussian_major: output arrays are null");
    const size_t wneed = gauss_major_work_bytes(nq);
    if (!work || work_bytes < wneed || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_sample_gaussian_major: workspace needs %zu bytes, 256-byte aligned (got %zu)",
                    wneed, work_bytes);
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
    Plan p;
    if ((st = order_queries("gs_sample_gaussian_major", qp, gp, nq, plan, plan_bytes, &p, stream)) != GS_OK)
        return st;
    GS_TRY(launch_sample_gauss_major(qp, gp, bwd_geom(gp, qp, cutoff_T(index->tau)), w.rec, w.box, w.gorder,
                                     index->n_gauss, p.order, p.point_off,
                                     cutoff_T(index->tau), index->tau, out_value, out_influence, p.res, work, stream),
           "gs_sample_gaussian_major");
    return GS_OK;
}

size_t gs_backward_work_bytes(const gs_index *index, const gs_query *query) {
    std::string why;
    if (!index || index->n_pairs < 0 || !query_valid(query, &why)) return (size_t)-1;
    return bwd_layout(nullptr, index, query).bytes;
}

gs_status gs_sample_backward(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                             const void *plan, size_t plan_bytes, const float *value, const float *influence,
                             const float *grad_value, const float *grad_influence, float *d_mean, float *d_scale,
                             float *d_rot, float *d_value, float *d_weight, void *work, size_t work_bytes,
                             hipStream_t stream) {
    gs_status st = check_index("gs_sample_backward", gauss, index);
    if (st != GS_OK) return st;
    if ((st = check_query("gs_sample_backward", index, query)) != GS_OK) return st;
    const int64_t n = gauss->n;
    const int64_t nq = query_count(query);
    if (nq > 0 && (!value || !influence || !grad_value || !grad_influence))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_backward: forward outputs or cotangents are null");
    if (n > 0 && (!d_mean || !d_scale || !d_rot || !d_value || !d_weight))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_backward: gradient arrays are null");
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    const size_t need = bwd_layout(nullptr, index, query).bytes;
    if (!work || work_bytes < need || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_sample_backward: workspace needs %zu bytes, 256-byte aligned (got %zu)",
                    need, work_bytes);
    Plan p{};
    if (query->kind != GS_QUERY_GRID) {
        const size_t pneed = plan_layout(nullptr, nq, gp.ncells).bytes;
        if (!plan || plan_bytes < pneed || !aligned(plan))
            return fail(GS_ERR_WORKSPACE, "gs_sample_backward: plan needs %zu bytes (got %zu)", pneed, plan_bytes);
        p = plan_layout(const_cast<void *>(plan), nq, gp.ncells);
    }
    IndexWork w = index_layout(index->work, n, &index->grid, index->capacity);
    BwdWork bw = bwd_layout(work, index, query);
    const float T = cutoff_T(index->tau);
    GS_TRY(launch_backward(qp, gp, bwd_geom(gp, qp, T), w.rec, w.box, w.gorder, n, index->n_pairs, p.order,
                           p.point_off, p.res.pos, p.res.out, value, influence, grad_value, grad_influence, T, bw.b,
                           gauss->scale, gauss->rot, d_mean, d_scale, d_rot, d_value, d_weight, stream),
           "gs_sample_backward");
    return GS_OK;
}

gs_status gs_sample_backward_noalloc(const gs_gaussians *gauss, const gs_index *index, const gs_query *query,
                                     const void *plan, size_t plan_bytes, const float *value, const float *influence,
                                     const float *grad_value, const float *grad_influence, float *d_mean,
                                     float *d_scale, float *d_rot, float *d_value, float *d_weight,
                                     hipStream_t stream) {
    std::string why;
    if (!index || index->n_pairs < 0 || !query_valid(query, &why))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_backward_noalloc: %s",
                    !index ? "index is null" : (index->n_pairs < 0 ? "the index has not been built" : why.c_str()));
    const size_t need = bwd_layout(nullptr, index, query).bytes;
    if (need > kNoAllocScratchBytes)
        return fail(GS_ERR_WORKSPACE,
                    "gs_sample_backward_noalloc: needs %zu bytes of workspace, more than its fixed %zu "
                    "(use gs_sample_backward with a workspace of gs_backward_work_bytes)",
                    need, kNoAllocScratchBytes);
    hipError_t e = hipSuccess;
    void *work = scratch_address(&e);
    if (!work) return hip_fail(e, "gs_sample_backward_noalloc: locating the static workspace");
    return gs_sample_backward(gauss, index, query, plan, plan_bytes, value, influence, grad_value, grad_influence,
                              d_mean, d_scale, d_rot, d_value, d_weight, work, kNoAllocScratchBytes, stream);
}

// ---------------------------------------------------------------------------
// Training epilogue (include/gs_train.h).

gs_status gs_activate(int64_t n, const float *log_scale, const float *value_logit, const float *weight_logit,
                      float scale_cap, float *scale, float *value, float *weight, hipStream_t stream) {
    if (n < 0 || n >= ((int64_t)1 << 31)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_activate: n = %lld out of range",
                                                      (long long)n);
    if (n == 0) return GS_OK;
    if (!log_scale || !value_logit || !weight_logit || !scale || !value || !weight)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_activate: null array");
    const double cap = std::isfinite(scale_cap) && scale_cap > 0.0f ? (double)scale_cap : 0.0;
    GS_TRY(launch_activate(n, log_scale, value_logit, weight_logit, cap, scale, value, weight, stream),
           "gs_activate");
    return GS_OK;
}

gs_status gs_activate_backward(int64_t n, const float *log_scale, const float *value_logit,
                               const float *weight_logit, float scale_cap, const float *d_scale,
                               const float *d_value, const float *d_weight, float *d_log_scale,
                               float *d_value_logit, float *d_weight_logit, hipStream_t stream) {
    if (n < 0 || n >= ((int64_t)1 << 31))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_activate_backward: n = %lld out of range", (long long)n);
    if (n == 0) return GS_OK;
    if (!log_scale || !value_logit || !weight_logit || !d_scale || !d_value || !d_weight || !d_log_scale ||
        !d_value_logit || !d_weight_logit)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_activate_backward: null array");
    const double cap = std::isfinite(scale_cap) && scale_cap > 0.0f ? (double)scale_cap : 0.0;
    GS_TRY(launch_activate_backward(n, log_scale, value_logit, weight_logit, cap, d_scale, d_value, d_weight,
                                    d_log_scale, d_value_logit, d_weight_logit, stream),
           "gs_activate_backward");
    return GS_OK;
}

size_t gs_loss_work_bytes(int64_t n) {
    if (n < 0 || n >= ((int64_t)1 << 31)) return (size_t)-1;
    return loss_work_bytes(n);
}

gs_status gs_loss(int64_t n, const float *value, const float *influence, const float *target,
                  const uint8_t *defined, const gs_loss_params *params, float *grad_value, float *grad_influence,
                  gs_loss_terms *terms, void *work, size_t work_bytes, hipStream_t stream) {
    if (n < 0 || n >= ((int64_t)1 << 31)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: n = %lld out of range",
                                                      (long long)n);
    if (!params || !terms) return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: params or terms is null");
    if (n > 0 && (!value || !influence || !target || !grad_value || !grad_influence))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: null array");
    const gs_loss_params p = *params;
    if (!(p.tau > 0.0f && p.tau < 1.0f)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: tau must lie in (0, 1)");
    if (!(std::isfinite(p.fn_eps) && p.fn_eps >= 0.0f))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: fn_eps must be finite and >= 0");
    if (!std::isfinite(p.fn_lambda) || !std::isfinite(p.fp_lambda))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_loss: loss weights must be finite");
    const size_t need = loss_work_bytes(n);
    if (!work || work_bytes < need || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_loss: workspace needs %zu bytes, 256-byte aligned (got %zu)", need,
                    work_bytes);
    GS_TRY(launch_loss(n, value, influence, target, defined, p.tau, p.fn_eps, p.fn_lambda, p.fp_lambda, grad_value,
                       grad_influence, terms, work, stream),
           "gs_loss");
    return GS_OK;
}

size_t gs_densify_work_bytes(int64_t n_in, const gs_query *query) {
    if (n_in < 0 || n_in >= ((int64_t)1 << 31)) return (size_t)-1;
    std::string why;
    if (!query_valid(query, &why)) return (size_t)-1;
    return densify_work_bytes(n_in, query_count(query));
}

gs_status gs_densify(const gs_params *in, int64_t n_in, const float *weight, const gs_grid *domain,
                     const gs_query *query, const float *value, const float *influence, const float *target,
                     const uint8_t *defined, const gs_densify_params *params, const gs_params *out,
                     int64_t capacity, int32_t *source, int64_t *n_out, void *work, size_t work_bytes,
                     hipStream_t stream) {
    if (!in || !out || !params || !n_out || !domain)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: null argument");
    *n_out = 0;
    if (n_in < 0 || n_in >= ((int64_t)1 << 31) || capacity < 0 || capacity >= ((int64_t)1 << 31))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: counts out of range");
    std::string why;
    if (!grid_valid(domain, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: %s", why.c_str());
    if (!query_valid(query, &why)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: %s", why.c_str());
    const int64_t nq = query_count(query);
    if (n_in > 0 && (!weight || !in->mean || !in->log_scale || !in->rot || !in->value_logit || !in->weight_logit))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: input arrays are null");
    if (capacity > 0 &&
        (!source || !out->mean || !out->log_scale || !out->rot || !out->value_logit || !out->weight_logit))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: output arrays are null");
    if (nq > 0 && (!value || !influence || !target))
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: forward outputs or targets are null");
    const gs_densify_params p = *params;
    if (!(p.tau > 0.0f && p.tau < 1.0f)) return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: tau must lie in (0, 1)");
    if (std::isnan(p.prune_weight) || !std::isfinite(p.new_log_scale) || !std::isfinite(p.new_weight_logit) ||
        p.max_new < 0)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_densify: invalid settings");
    const size_t need = densify_work_bytes(n_in, nq);
    if (!work || work_bytes < need || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_densify: workspace needs %zu bytes, 256-byte aligned (got %zu)", need,
                    work_bytes);
    PinnedCount *pc = pinned_count();
    if (!pc) return fail(GS_ERR_HIP, "gs_densify: could not allocate the pinned read-back word");
    const GridParams gp = grid_params(domain);
    const QueryParams qp = query_params(query, domain);
    long long *n_out_dev = nullptr;
    GS_TRY(launch_densify(*in, n_in, weight, p.prune_weight, qp, gp, value, influence, target, defined, p.tau,
                          p.new_log_scale, p.new_weight_logit, p.max_new, capacity, *out, source, work, &n_out_dev,
                          stream),
           "gs_densify");
    GS_TRY(hipMemcpyAsync(pc->value, n_out_dev, sizeof(uint64_t), hipMemcpyDeviceToHost, stream),
           "gs_densify: count read-back");
    GS_TRY(hipEventRecord(pc->copied, stream), "gs_densify: event");
    GS_TRY(hipEventSynchronize(pc->copied), "gs_densify: wait");
    *n_out = (int64_t)*pc->value;
    if (*n_out > capacity)
        return fail(GS_ERR_CAPACITY, "gs_densify: %lld kept Gaussians exceed the capacity %lld", (long long)*n_out,
                    (long long)capacity);
    return GS_OK;
}

gs_status gs_backward_pair_count(const gs_index *index, const gs_query *query, const void *plan,
                                 size_t plan_bytes, void *work, size_t work_bytes, int64_t *count,
                                 hipStream_t stream) {
    if (!count) return fail(GS_ERR_INVALID_ARGUMENT, "gs_backward_pair_count: count is null");
    *count = 0;
    if (!index || index->n_pairs < 0 || index->n_gauss < 0)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_backward_pair_count: index not built");
    gs_status st = check_query("gs_backward_pair_count", index, query);
    if (st != GS_OK) return st;
    const int64_t nq = query_count(query);
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    const size_t need = bwd_layout(nullptr, index, query).bytes;
    if (!work || work_bytes < need || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_backward_pair_count: workspace needs %zu bytes (got %zu)", need,
                    work_bytes);
    Plan p{};
    if (query->kind != GS_QUERY_GRID) {
        const size_t pneed = plan_layout(nullptr, nq, gp.ncells).bytes;
        if (!plan || plan_bytes < pneed || !aligned(plan))
            return fail(GS_ERR_WORKSPACE, "gs_backward_pair_count: plan needs %zu bytes (got %zu)", pneed,
                        plan_bytes);
        p = plan_layout(const_cast<void *>(plan), nq, gp.ncells);
    }
    PinnedCount *pc = pinned_count();
    if (!pc) return fail(GS_ERR_HIP, "gs_backward_pair_count: could not allocate the pinned read-back word");
    IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
    BwdWork bw = bwd_layout(work, index, query);
    unsigned long long *total = (unsigned long long *)bw.b.moments;
    GS_TRY(launch_count_backward_pairs(qp, gp, bwd_geom(gp, qp, cutoff_T(index->tau)), w.rec, w.box,
                                       index->n_gauss, p.point_off, total, stream),
           "gs_backward_pair_count");
    GS_TRY(hipMemcpyAsync(pc->value, total, sizeof(uint64_t), hipMemcpyDeviceToHost, stream),
           "gs_backward_pair_count: read-back");
    GS_TRY(hipEventRecord(pc->copied, stream), "gs_backward_pair_count: event");
    GS_TRY(hipEventSynchronize(pc->copied), "gs_backward_pair_count: wait");
    *count = (int64_t)*pc->value;
    return GS_OK;
}

gs_status gs_sample_pair_counts(const gs_index *index, const gs_query *query, const void *plan, size_t plan_bytes,
                                void *work, size_t work_bytes, int64_t *tests, int64_t *contributing,
                                hipStream_t stream) {
    if (!tests || !contributing)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_pair_counts: output counts are null");
    *tests = *contributing = 0;
    if (!index || index->n_pairs < 0 || index->n_pairs > index->capacity || index->n_gauss < 0 || !index->work ||
        !index->cell_offsets)
        return fail(GS_ERR_INVALID_ARGUMENT, "gs_sample_pair_counts: index not built");
    gs_status st = check_query("gs_sample_pair_counts", index, query);
    if (st != GS_OK) return st;
    const int64_t nq = query_count(query);
    const GridParams gp = grid_params(&index->grid);
    const QueryParams qp = query_params(query, &index->grid);
    const size_t need = bwd_layout(nullptr, index, query).bytes;
    if (!work || work_bytes < need || !aligned(work))
        return fail(GS_ERR_WORKSPACE, "gs_sample_pair_counts: workspace needs %zu bytes (got %zu)", need, work_bytes);
    Plan p{};
    if (query->kind != GS_QUERY_GRID) {
        const size_t pneed = plan_layout(nullptr, nq, gp.ncells).bytes;
        if (!plan || plan_bytes < pneed || !aligned(plan))
            return fail(GS_ERR_WORKSPACE, "gs_sample_pair_counts: plan needs %zu bytes (got %zu)", pneed,
                        plan_bytes);
        p = plan_layout(const_cast<void *>(plan), nq, gp.ncells);
    }
    PinnedCount *pc = pinned_count();
    if (!pc) return fail(GS_ERR_HIP, "gs_sample_pair_counts: could not allocate the pinned read-back word");
    IndexWork w = index_layout(index->work, index->n_gauss, &index->grid, index->capacity);
    BwdWork bw = bwd_layout(work, index, query);
    unsigned long long *totals = (unsigned long long *)bw.b.moments;
    GS_TRY(launch_count_sample_pairs(qp, gp, w.rec, index->gids, index->cell_offsets, p.keys, p.res.pos,
                                     cutoff_T(index->tau), totals, stream),
           "gs_sample_pair_counts");
    for (int k = 0; k < 2; ++k) {
        GS_TRY(hipMemcpyAsync(pc->value, totals + k, sizeof(uint64_t), hipMemcpyDeviceToHost, stream),
               "gs_sample_pair_counts: read-back");
        GS_TRY(hipEventRecord(pc->copied, stream), "gs_sample_pair_counts: event");
        GS_TRY(hipEventSynchronize(pc->copied), "gs_sample_pair_counts: wait");
        (k == 0 ? *tests : *contributing) = (int64_t)*pc->value;
    }
    return GS_OK;
}

}  // extern "C"
