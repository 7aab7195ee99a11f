"""Python binding of the C-ABI in include/gs.h and include/gs_train.h (ctypes).

Argument marshalling only: every step of sampling runs in the HIP library
libgsq.so. torch provides device memory and the stream. Importing this module
does not touch the GPU; the first call loads the library and raises
GsLibraryMissing if it has not been built (python -m
paper_2607_01164_amd.build) -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgsq.so")

GS_OK = 0
GS_ERR_INVALID_ARGUMENT = 1
GS_ERR_CAPACITY = 2
GS_ERR_WORKSPACE = 3
GS_ERR_HIP = 4

GS_QUERY_GRID = 0
GS_QUERY_VOXELS = 1
GS_QUERY_POINTS = 2
GS_QUERY_JITTER = 3

EXPORTED = ("gs_query_size", "gs_index_work_bytes", "gs_build_index", "gs_plan_bytes", "gs_sample",
            "gs_backward_work_bytes", "gs_sample_backward", "gs_last_error", "gs_version", "gs_profile_enable",
            "gs_profile_select", "gs_profile_reset", "gs_profile_read", "gs_activate", "gs_activate_backward",
            "gs_loss_work_bytes", "gs_loss", "gs_densify_work_bytes", "gs_densify",
            "gs_sample_gaussian_major_work_bytes", "gs_sample_gaussian_major", "gs_backward_pair_count",
            "gs_sample_pair_counts", "gs_sample_backward_noalloc", "gs_plan_queries", "gs_sample_planned")


class GsLibraryMissing(RuntimeError):
    pass


class GsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[gs status {status}] {message}")
        self.status = status


class GsGaussians(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("mean", ctypes.c_void_p), ("scale", ctypes.c_void_p),
                ("rot", ctypes.c_void_p), ("value", ctypes.c_void_p), ("weight", ctypes.c_void_p)]


class GsGrid(ctypes.Structure):
    _fields_ = [("lo", ctypes.c_float * 3), ("hi", ctypes.c_float * 3), ("cells", ctypes.c_int32 * 3)]


class GsIndex(ctypes.Structure):
    _fields_ = [("keys", ctypes.c_void_p), ("gids", ctypes.c_void_p), ("cell_offsets", ctypes.c_void_p),
                ("capacity", ctypes.c_int64), ("work", ctypes.c_void_p), ("work_bytes", ctypes.c_size_t),
                ("n_pairs", ctypes.c_int64), ("n_gauss", ctypes.c_int64), ("grid", GsGrid), ("tau", ctypes.c_float)]


class GsQuery(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dims", ctypes.c_int32 * 3), ("n", ctypes.c_int64),
                ("voxel_ids", ctypes.c_void_p), ("points", ctypes.c_void_p)]


class GsLossParams(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("fn_eps", ctypes.c_float), ("fn_lambda", ctypes.c_float),
                ("fp_lambda", ctypes.c_float)]


class GsParams(ctypes.Structure):
    _fields_ = [("mean", ctypes.c_void_p), ("log_scale", ctypes.c_void_p), ("rot", ctypes.c_void_p),
                ("value_logit", ctypes.c_void_p), ("weight_logit", ctypes.c_void_p)]


class GsDensifyParams(ctypes.Structure):
    _fields_ = [("prune_weight", ctypes.c_float), ("tau", ctypes.c_float), ("new_log_scale", ctypes.c_float),
                ("new_weight_logit", ctypes.c_float), ("max_new", ctypes.c_int64)]


LOSS_TERMS_BYTES = 64  # gs_loss_terms: four float64 values, then four int64 counts

_LIB = None


def load_library():
    """Load libgsq.so (built in-tree) and declare the exported signatures."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise GsLibraryMissing(f"{LIB_PATH} is missing: build it with `python -m paper_2607_01164_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    L.gs_query_size.restype = i64
    L.gs_query_size.argtypes = [P(GsQuery)]
    L.gs_index_work_bytes.restype = sz
    L.gs_index_work_bytes.argtypes = [i64, P(GsGrid), i64]
    L.gs_build_index.restype = ctypes.c_int
    L.gs_build_index.argtypes = [P(GsGaussians), P(GsGrid), ctypes.c_float, P(GsIndex), vp]
    L.gs_plan_bytes.restype = sz
    L.gs_plan_bytes.argtypes = [P(GsQuery), P(GsGrid)]
    L.gs_sample.restype = ctypes.c_int
    L.gs_sample.argtypes = [P(GsGaussians), P(GsIndex), P(GsQuery), vp, vp, vp, sz, vp]
    L.gs_plan_queries.restype = ctypes.c_int
    L.gs_plan_queries.argtypes = [P(GsQuery), P(GsGrid), vp, sz, vp]
    L.gs_sample_planned.restype = ctypes.c_int
    L.gs_sample_planned.argtypes = [P(GsGaussians), P(GsIndex), P(GsQuery), vp, vp, vp, sz, vp]
    L.gs_sample_gaussian_major_work_bytes.restype = sz
    L.gs_sample_gaussian_major_work_bytes.argtypes = [P(GsQuery)]
    L.gs_sample_gaussian_major.restype = ctypes.c_int
    L.gs_sample_gaussian_major.argtypes = [P(GsGaussians), P(GsIndex), P(GsQuery), vp, vp, vp, sz, vp, sz, vp]
    L.gs_backward_pair_count.restype = ctypes.c_int
    L.gs_backward_pair_count.argtypes = [P(GsIndex), P(GsQuery), vp, sz, vp, sz, P(i64), vp]
    L.gs_sample_pair_counts.restype = ctypes.c_int
    L.gs_sample_pair_counts.argtypes = [P(GsIndex), P(GsQuery), vp, sz, vp, sz, P(i64), P(i64), vp]
    L.gs_backward_work_bytes.restype = sz
    L.gs_backward_work_bytes.argtypes = [P(GsIndex), P(GsQuery)]
    L.gs_sample_backward.restype = ctypes.c_int
    L.gs_sample_backward.argtypes = [P(GsGaussians), P(GsIndex), P(GsQuery), vp, sz, vp, vp, vp, vp, vp, vp, vp, vp,
                                     vp, vp, sz, vp]
    L.gs_sample_backward_noalloc.restype = ctypes.c_int
    L.gs_sample_backward_noalloc.argtypes = [P(GsGaussians), P(GsIndex), P(GsQuery), vp, sz, vp, vp, vp, vp, vp,
                                             vp, vp, vp, vp, vp]
    L.gs_last_error.restype = ctypes.c_char_p
    L.gs_last_error.argtypes = []
    L.gs_version.restype = ctypes.c_int
    L.gs_version.argtypes = []
    L.gs_profile_enable.restype = None
    L.gs_profile_enable.argtypes = [ctypes.c_int]
    L.gs_profile_select.restype = None
    L.gs_profile_select.argtypes = [ctypes.c_char_p]
    L.gs_profile_reset.restype = None
    L.gs_profile_reset.argtypes = []
    L.gs_profile_read.restype = ctypes.c_int
    L.gs_profile_read.argtypes = [P(ctypes.c_char_p), P(i64), P(ctypes.c_double), ctypes.c_int]
    f32 = ctypes.c_float
    L.gs_activate.restype = ctypes.c_int
    L.gs_activate.argtypes = [i64, vp, vp, vp, f32, vp, vp, vp, vp]
    L.gs_activate_backward.restype = ctypes.c_int
    L.gs_activate_backward.argtypes = [i64, vp, vp, vp, f32, vp, vp, vp, vp, vp, vp, vp]
    L.gs_loss_work_bytes.restype = sz
    L.gs_loss_work_bytes.argtypes = [i64]
    L.gs_loss.restype = ctypes.c_int
    L.gs_loss.argtypes = [i64, vp, vp, vp, vp, P(GsLossParams), vp, vp, vp, vp, sz, vp]
    L.gs_densify_work_bytes.restype = sz
    L.gs_densify_work_bytes.argtypes = [i64, P(GsQuery)]
    L.gs_densify.restype = ctypes.c_int
    L.gs_densify.argtypes = [P(GsParams), i64, vp, P(GsGrid), P(GsQuery), vp, vp, vp, vp, P(GsDensifyParams),
                             P(GsParams), i64, vp, P(i64), vp, sz, vp]
    _LIB = L
    return L


def _check(status: int):
    if status != GS_OK:
        msg = load_library().gs_last_error().decode(errors="replace")
        raise GsError(status, msg)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_f32(t: torch.Tensor, name: str, shape_tail=()) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous float32")
    if shape_tail and tuple(t.shape[1:]) != tuple(shape_tail):
        raise ValueError(f"{name} must have shape [n, {', '.join(map(str, shape_tail))}]")
    return t


@dataclass
class Gaussians:
    """Post-activation parameters on the device: mean [n,3], scale [n,3],
    rot [n,4] (w,x,y,z), value [n], weight [n]."""
    mean: torch.Tensor
    scale: torch.Tensor
    rot: torch.Tensor
    value: torch.Tensor
    weight: torch.Tensor

    @property
    def n(self) -> int:
        return int(self.mean.shape[0])

    def c(self) -> GsGaussians:
        n = self.n
        _dev_f32(self.mean, "mean", (3,))
        _dev_f32(self.scale, "scale", (3,))
        _dev_f32(self.rot, "rot", (4,))
        _dev_f32(self.value, "value")
        _dev_f32(self.weight, "weight")
        for t in (self.scale, self.rot):
            if t.shape[0] != n:
                raise ValueError("parameter arrays disagree on n")
        for t in (self.value, self.weight):
            if t.numel() != n:
                raise ValueError("parameter arrays disagree on n")
        return GsGaussians(n, self.mean.data_ptr(), self.scale.data_ptr(), self.rot.data_ptr(),
                           self.value.data_ptr(), self.weight.data_ptr())


def make_grid(cells: Sequence[int], lo=(0.0, 0.0, 0.0), hi=(1.0, 1.0, 1.0)) -> GsGrid:
    return GsGrid((ctypes.c_float * 3)(*lo), (ctypes.c_float * 3)(*hi), (ctypes.c_int32 * 3)(*cells))


@dataclass
class Query:
    kind: int
    dims: Sequence[int] = (0, 0, 0)
    voxel_ids: Optional[torch.Tensor] = None  # uint32 stored as int32 [n]
    points: Optional[torch.Tensor] = None     # float32 [n,3]

    @staticmethod
    def grid(dims) -> "Query":
        return Query(GS_QUERY_GRID, tuple(dims))

    @staticmethod
    def voxels(dims, ids: torch.Tensor) -> "Query":
        return Query(GS_QUERY_VOXELS, tuple(dims), voxel_ids=ids)

    @staticmethod
    def pts(points: torch.Tensor) -> "Query":
        return Query(GS_QUERY_POINTS, (0, 0, 0), points=points)

    @staticmethod
    def jitter(dims, offsets: torch.Tensor, ids: Optional[torch.Tensor] = None) -> "Query":
        """One position per voxel at lo + (i + u) * voxel size: offsets u
        [n, 3] (in [0, 1) for a position inside the voxel), for the listed
        voxel ids, or for every voxel (x fastest) when ids is None."""
        return Query(GS_QUERY_JITTER, tuple(dims), voxel_ids=ids, points=offsets)

    def c(self) -> GsQuery:
        n = 0
        if self.kind == GS_QUERY_VOXELS or (self.kind == GS_QUERY_JITTER and self.voxel_ids is not None):
            if self.voxel_ids is None or not self.voxel_ids.is_cuda or self.voxel_ids.element_size() != 4 or \
                    not self.voxel_ids.is_contiguous():
                raise ValueError("voxel_ids must be a contiguous 32-bit device tensor")
            n = self.voxel_ids.numel()
        if self.kind == GS_QUERY_POINTS:
            _dev_f32(self.points, "points", (3,))
            n = self.points.shape[0]
        elif self.kind == GS_QUERY_JITTER:
            _dev_f32(self.points, "jitter offsets", (3,))
            if self.voxel_ids is None:
                n = self.points.shape[0]
            elif self.points.shape[0] != n:
                raise ValueError("jitter offsets must have one row per voxel id")
        d = tuple(self.dims) if self.kind != GS_QUERY_POINTS else (0, 0, 0)
        return GsQuery(self.kind, (ctypes.c_int32 * 3)(*d), n, _ptr(self.voxel_ids), _ptr(self.points))

    def size(self) -> int:
        q = self.c()
        return int(load_library().gs_query_size(ctypes.byref(q)))


def _alloc_bytes(nbytes: int, device) -> torch.Tensor:
    # 256-byte alignment: torch's caching allocator returns 512-byte aligned blocks
    t = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    assert t.data_ptr() % 256 == 0
    return t


class Index:
    """A built cell index: owns its device buffers (torch tensors) and the
    C struct that points at them."""

    def __init__(self, grid: GsGrid, n_gauss: int, capacity: int, device):
        L = load_library()
        self.grid = grid
        self.capacity = int(capacity)
        self.device = device
        ncells = grid.cells[0] * grid.cells[1] * grid.cells[2]
        self.keys = torch.empty(max(self.capacity, 1), dtype=torch.int32, device=device)
        self.gids = torch.empty(max(self.capacity, 1), dtype=torch.int32, device=device)
        self.cell_offsets = torch.empty(ncells + 1, dtype=torch.int32, device=device)
        wb = L.gs_index_work_bytes(n_gauss, ctypes.byref(grid), self.capacity)
        if wb == ctypes.c_size_t(-1).value:
            raise GsError(GS_ERR_INVALID_ARGUMENT, "bad grid or sizes")
        self.work = _alloc_bytes(wb, device)
        self.c = GsIndex(self.keys.data_ptr(), self.gids.data_ptr(), self.cell_offsets.data_ptr(), self.capacity,
                         self.work.data_ptr(), int(self.work.numel()), -1, 0, grid, 0.0)

    @property
    def n_pairs(self) -> int:
        return int(self.c.n_pairs)


def gs_build_index(gauss: Gaussians, grid: GsGrid, tau: float, index: Index, stream=None) -> int:
    """Build the index into `index`; raises GsError (status GS_ERR_CAPACITY
    with index.n_pairs set when the capacity is too small)."""
    g = gauss.c()
    st = load_library().gs_build_index(ctypes.byref(g), ctypes.byref(grid), float(tau), ctypes.byref(index.c),
                                       _stream(stream))
    _check(st)
    return index.n_pairs


def build_index(gauss: Gaussians, grid: GsGrid, tau: float = 0.01, capacity: Optional[int] = None,
                stream=None) -> Index:
    """Allocate and build an index, growing the pair capacity once if needed."""
    dev = gauss.mean.device
    cap = int(capacity) if capacity is not None else max(1 << 16, 64 * gauss.n)
    idx = Index(grid, gauss.n, cap, dev)
    try:
        gs_build_index(gauss, grid, tau, idx, stream)
    except GsError as e:
        if e.status != GS_ERR_CAPACITY:
            raise
        need = idx.n_pairs
        idx = Index(grid, gauss.n, int(need * 1.05) + 1024, dev)
        gs_build_index(gauss, grid, tau, idx, stream)
    return idx


def plan_bytes(query: Query, grid: GsGrid) -> int:
    q = query.c()
    b = load_library().gs_plan_bytes(ctypes.byref(q), ctypes.byref(grid))
    if b == ctypes.c_size_t(-1).value:
        raise GsError(GS_ERR_INVALID_ARGUMENT, "malformed query or grid")
    return int(b)


def alloc_plan(query: Query, grid: GsGrid, device) -> torch.Tensor:
    return _alloc_bytes(plan_bytes(query, grid), device)


def gs_sample(gauss: Gaussians, index: Index, query: Query, out_value: torch.Tensor, out_influence: torch.Tensor,
              plan: Optional[torch.Tensor] = None, stream=None) -> None:
    g = gauss.c()
    q = query.c()
    n = query.size()
    for t, nm in ((out_value, "out_value"), (out_influence, "out_influence")):
        _dev_f32(t, nm)
        if t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements")
    st = load_library().gs_sample(ctypes.byref(g), ctypes.byref(index.c), ctypes.byref(q), out_value.data_ptr(),
                                  out_influence.data_ptr(), _ptr(plan), 0 if plan is None else plan.numel(),
                                  _stream(stream))
    _check(st)


def gs_plan_queries(query: Query, grid: GsGrid, plan: Optional[torch.Tensor], stream=None) -> None:
    """The query ordering of gs_sample alone, for gs_sample_planned (it may
    run on another stream than the index build)."""
    q = query.c()
    st = load_library().gs_plan_queries(ctypes.byref(q), ctypes.byref(grid), _ptr(plan),
                                        0 if plan is None else plan.numel(), _stream(stream))
    _check(st)


def gs_sample_planned(gauss: Gaussians, index: Index, query: Query, out_value: torch.Tensor,
                      out_influence: torch.Tensor, plan: Optional[torch.Tensor] = None, stream=None) -> None:
    """gs_sample with a plan that gs_plan_queries filled for this query and
    the index's grid."""
    g = gauss.c()
    q = query.c()
    n = query.size()
    for t, nm in ((out_value, "out_value"), (out_influence, "out_influence")):
        _dev_f32(t, nm)
        if t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements")
    st = load_library().gs_sample_planned(ctypes.byref(g), ctypes.byref(index.c), ctypes.byref(q),
                                          out_value.data_ptr(), out_influence.data_ptr(), _ptr(plan),
                                          0 if plan is None else plan.numel(), _stream(stream))
    _check(st)


def gaussian_major_work_bytes(query: Query) -> int:
    q = query.c()
    b = load_library().gs_sample_gaussian_major_work_bytes(ctypes.byref(q))
    if b == ctypes.c_size_t(-1).value:
        raise GsError(GS_ERR_INVALID_ARGUMENT, "grid or malformed query")
    return int(b)


def alloc_gaussian_major_work(query: Query, device) -> torch.Tensor:
    return _alloc_bytes(gaussian_major_work_bytes(query), device)


def gs_sample_gaussian_major(gauss: Gaussians, index: Index, query: Query, out_value: torch.Tensor,
                             out_influence: torch.Tensor, plan: torch.Tensor, work: torch.Tensor, stream=None) -> None:
    """The paper's Gaussian-major forward (Sec. 5.1.2) as a variant of
    gs_sample for voxel-list, point and jittered queries."""
    g = gauss.c()
    q = query.c()
    n = query.size()
    for t, nm in ((out_value, "out_value"), (out_influence, "out_influence")):
        _dev_f32(t, nm)
        if t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements")
    st = load_library().gs_sample_gaussian_major(ctypes.byref(g), ctypes.byref(index.c), ctypes.byref(q),
                                                 out_value.data_ptr(), out_influence.data_ptr(), _ptr(plan),
                                                 0 if plan is None else plan.numel(), _ptr(work),
                                                 0 if work is None else work.numel(), _stream(stream))
    _check(st)


def backward_work_bytes(index: Index, query: Query) -> int:
    q = query.c()
    b = load_library().gs_backward_work_bytes(ctypes.byref(index.c), ctypes.byref(q))
    if b == ctypes.c_size_t(-1).value:
        raise GsError(GS_ERR_INVALID_ARGUMENT, "index not built or malformed query")
    return int(b)


def alloc_backward_work(index: Index, query: Query, device) -> torch.Tensor:
    return _alloc_bytes(backward_work_bytes(index, query), device)


@dataclass
class Grads:
    mean: torch.Tensor
    scale: torch.Tensor
    rot: torch.Tensor
    value: torch.Tensor
    weight: torch.Tensor

    @staticmethod
    def empty(n: int, device) -> "Grads":
        f = dict(dtype=torch.float32, device=device)
        return Grads(torch.empty(n, 3, **f), torch.empty(n, 3, **f), torch.empty(n, 4, **f), torch.empty(n, **f),
                     torch.empty(n, **f))


def gs_sample_backward(gauss: Gaussians, index: Index, query: Query, plan: Optional[torch.Tensor],
                       value: torch.Tensor, influence: torch.Tensor, grad_value: torch.Tensor,
                       grad_influence: torch.Tensor, grads: Grads, work: torch.Tensor, stream=None) -> None:
    g = gauss.c()
    q = query.c()
    n = query.size()
    for t, nm in ((value, "value"), (influence, "influence"), (grad_value, "grad_value"),
                  (grad_influence, "grad_influence")):
        _dev_f32(t, nm)
        if t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements")
    for t, nm in ((grads.mean, "d_mean"), (grads.scale, "d_scale"), (grads.rot, "d_rot"), (grads.value, "d_value"),
                  (grads.weight, "d_weight")):
        _dev_f32(t, nm)
    st = load_library().gs_sample_backward(
        ctypes.byref(g), ctypes.byref(index.c), ctypes.byref(q), _ptr(plan), 0 if plan is None else plan.numel(),
        value.data_ptr(), influence.data_ptr(), grad_value.data_ptr(), grad_influence.data_ptr(),
        grads.mean.data_ptr(), grads.scale.data_ptr(), grads.rot.data_ptr(), grads.value.data_ptr(),
        grads.weight.data_ptr(), work.data_ptr(), work.numel(), _stream(stream))
    _check(st)


def gs_sample_backward_noalloc(gauss: Gaussians, index: Index, query: Query, plan: Optional[torch.Tensor],
                               value: torch.Tensor, influence: torch.Tensor, grad_value: torch.Tensor,
                               grad_influence: torch.Tensor, grads: Grads, stream=None) -> None:
    """gs_sample_backward with the library's static workspace (no device
    allocation; see include/gs.h)."""
    g = gauss.c()
    q = query.c()
    n = query.size()
    for t, nm in ((value, "value"), (influence, "influence"), (grad_value, "grad_value"),
                  (grad_influence, "grad_influence")):
        _dev_f32(t, nm)
        if t.numel() < n:
            raise ValueError(f"{nm} needs {n} elements")
    for t, nm in ((grads.mean, "d_mean"), (grads.scale, "d_scale"), (grads.rot, "d_rot"), (grads.value, "d_value"),
                  (grads.weight, "d_weight")):
        _dev_f32(t, nm)
    st = load_library().gs_sample_backward_noalloc(
        ctypes.byref(g), ctypes.byref(index.c), ctypes.byref(q), _ptr(plan), 0 if plan is None else plan.numel(),
        value.data_ptr(), influence.data_ptr(), grad_value.data_ptr(), grad_influence.data_ptr(),
        grads.mean.data_ptr(), grads.scale.data_ptr(), grads.rot.data_ptr(), grads.value.data_ptr(),
        grads.weight.data_ptr(), _stream(stream))
    _check(st)


@dataclass
class RawParams:
    """Free parameters before the activations of Sec. 4.2: log_scale [n,3],
    value_logit [n], weight_logit [n] (means and quaternions are used as
    they are)."""
    log_scale: torch.Tensor
    value_logit: torch.Tensor
    weight_logit: torch.Tensor

    @property
    def n(self) -> int:
        return int(self.log_scale.shape[0])

    def check(self):
        _dev_f32(self.log_scale, "log_scale", (3,))
        for t, nm in ((self.value_logit, "value_logit"), (self.weight_logit, "weight_logit")):
            _dev_f32(t, nm)
            if t.numel() != self.n:
                raise ValueError("parameter arrays disagree on n")


def gs_activate(raw: RawParams, scale_cap: float, scale: torch.Tensor, value: torch.Tensor, weight: torch.Tensor,
                stream=None) -> None:
    raw.check()
    n = raw.n
    _dev_f32(scale, "scale", (3,))
    for t, nm in ((value, "value"), (weight, "weight")):
        _dev_f32(t, nm)
    if scale.shape[0] != n or value.numel() != n or weight.numel() != n:
        raise ValueError("output arrays must hold n Gaussians")
    st = load_library().gs_activate(n, raw.log_scale.data_ptr(), raw.value_logit.data_ptr(),
                                    raw.weight_logit.data_ptr(), float(scale_cap), scale.data_ptr(),
                                    value.data_ptr(), weight.data_ptr(), _stream(stream))
    _check(st)


def gs_activate_backward(raw: RawParams, scale_cap: float, grads: "Grads", out: RawParams, stream=None) -> None:
    """Gradients of the free parameters (into out) from grads, the
    gradients of the activated scale, value and weight."""
    raw.check()
    out.check()
    n = raw.n
    for t, nm in ((grads.scale, "d_scale"), (grads.value, "d_value"), (grads.weight, "d_weight")):
        _dev_f32(t, nm)
        if t.shape[0] != n:
            raise ValueError(f"{nm} must hold n Gaussians")
    if out.n != n:
        raise ValueError("output arrays must hold n Gaussians")
    st = load_library().gs_activate_backward(
        n, raw.log_scale.data_ptr(), raw.value_logit.data_ptr(), raw.weight_logit.data_ptr(), float(scale_cap),
        grads.scale.data_ptr(), grads.value.data_ptr(), grads.weight.data_ptr(), out.log_scale.data_ptr(),
        out.value_logit.data_ptr(), out.weight_logit.data_ptr(), _stream(stream))
    _check(st)


def loss_work_bytes(n: int) -> int:
    b = load_library().gs_loss_work_bytes(int(n))
    if b == ctypes.c_size_t(-1).value:
        raise GsError(GS_ERR_INVALID_ARGUMENT, f"batch size {n} out of range")
    return int(b)


def alloc_loss_work(n: int, device) -> torch.Tensor:
    return _alloc_bytes(loss_work_bytes(n), device)


def alloc_loss_terms(device) -> torch.Tensor:
    return torch.zeros(LOSS_TERMS_BYTES, dtype=torch.uint8, device=device)


def read_loss_terms(terms: torch.Tensor) -> dict:
    """The gs_loss_terms a gs_loss call wrote (copies to the host)."""
    b = terms.cpu()
    d = b[:32].view(torch.float64).tolist()
    c = b[32:64].view(torch.int64).tolist()
    return {"l1": d[0], "fn": d[1], "fp": d[2], "total": d[3], "n_defined": c[0], "n_fn": c[1], "n_fp": c[2],
            "n": c[3]}


def gs_loss(value: torch.Tensor, influence: torch.Tensor, target: torch.Tensor, defined: Optional[torch.Tensor],
            tau: float, fn_eps: float, fn_lambda: float, fp_lambda: float, grad_value: torch.Tensor,
            grad_influence: torch.Tensor, terms: torch.Tensor, work: torch.Tensor, stream=None) -> None:
    """L1 + false-negative (Eq. 4) + false-positive (Eq. 5) losses of a
    batch and their cotangents; defined is a uint8 flag per sample (None:
    every sample lies in the volume). terms: LOSS_TERMS_BYTES device bytes."""
    n = int(value.numel())
    for t, nm in ((value, "value"), (influence, "influence"), (target, "target"), (grad_value, "grad_value"),
                  (grad_influence, "grad_influence")):
        _dev_f32(t, nm)
        if t.numel() != n:
            raise ValueError(f"{nm} must have {n} elements")
    if defined is not None:
        if not defined.is_cuda or defined.dtype != torch.uint8 or not defined.is_contiguous() or defined.numel() != n:
            raise ValueError("defined must be a contiguous uint8 device tensor of n elements")
    if not terms.is_cuda or terms.numel() * terms.element_size() < LOSS_TERMS_BYTES or terms.data_ptr() % 8:
        raise ValueError("terms must be a device buffer of at least 64 bytes, 8-byte aligned")
    p = GsLossParams(float(tau), float(fn_eps), float(fn_lambda), float(fp_lambda))
    st = load_library().gs_loss(n, value.data_ptr(), influence.data_ptr(), target.data_ptr(), _ptr(defined),
                                ctypes.byref(p), grad_value.data_ptr(), grad_influence.data_ptr(), terms.data_ptr(),
                                work.data_ptr(), work.numel() * work.element_size(), _stream(stream))
    _check(st)


@dataclass
class ParamSet:
    """Free parameters of up to `rows` Gaussians on the device: mean [rows,3],
    log_scale [rows,3], rot [rows,4], value_logit [rows], weight_logit
    [rows]."""
    mean: torch.Tensor
    log_scale: torch.Tensor
    rot: torch.Tensor
    value_logit: torch.Tensor
    weight_logit: torch.Tensor

    @staticmethod
    def empty(rows: int, device) -> "ParamSet":
        f = dict(dtype=torch.float32, device=device)
        return ParamSet(torch.empty(rows, 3, **f), torch.empty(rows, 3, **f), torch.empty(rows, 4, **f),
                        torch.empty(rows, **f), torch.empty(rows, **f))

    @property
    def rows(self) -> int:
        return int(self.mean.shape[0])

    def c(self) -> GsParams:
        r = self.rows
        for t, nm, tail in ((self.mean, "mean", (3,)), (self.log_scale, "log_scale", (3,)), (self.rot, "rot", (4,)),
                            (self.value_logit, "value_logit", ()), (self.weight_logit, "weight_logit", ())):
            _dev_f32(t, nm, tail)
            if t.shape[0] != r:
                raise ValueError("parameter arrays disagree on their rows")
        return GsParams(self.mean.data_ptr(), self.log_scale.data_ptr(), self.rot.data_ptr(),
                        self.value_logit.data_ptr(), self.weight_logit.data_ptr())

    def raw(self, n: Optional[int] = None) -> RawParams:
        n = self.rows if n is None else n
        return RawParams(self.log_scale[:n], self.value_logit[:n], self.weight_logit[:n])


def densify_work_bytes(n_in: int, query: Query) -> int:
    q = query.c()
    b = load_library().gs_densify_work_bytes(int(n_in), ctypes.byref(q))
    if b == ctypes.c_size_t(-1).value:
        raise GsError(GS_ERR_INVALID_ARGUMENT, "malformed query or count")
    return int(b)


def alloc_densify_work(n_in: int, query: Query, device) -> torch.Tensor:
    return _alloc_bytes(densify_work_bytes(n_in, query), device)


def gs_densify(params_in: ParamSet, n_in: int, weight: torch.Tensor, domain: GsGrid, query: Query,
               value: torch.Tensor, influence: torch.Tensor, target: torch.Tensor, defined: Optional[torch.Tensor],
               prune_weight: float, tau: float, new_log_scale: float, new_weight_logit: float, max_new: int,
               params_out: ParamSet, source: torch.Tensor, work: torch.Tensor, stream=None) -> int:
    """Weight pruning and sample-error densification (Sec. 4.2.1): writes the
    kept and new Gaussians into params_out (capacity = its rows) and the
    source map, and returns the new count (waits for it)."""
    nq = query.size()
    q = query.c()
    if n_in > params_in.rows:
        raise ValueError("n_in exceeds the input rows")
    _dev_f32(weight, "weight")
    if weight.numel() < n_in:
        raise ValueError("weight needs n_in elements")
    for t, nm in ((value, "value"), (influence, "influence"), (target, "target")):
        _dev_f32(t, nm)
        if t.numel() < nq:
            raise ValueError(f"{nm} needs {nq} elements")
    if defined is not None and (not defined.is_cuda or defined.dtype != torch.uint8 or defined.numel() < nq):
        raise ValueError("defined must be a uint8 device tensor of the query's size")
    cap = params_out.rows
    if not source.is_cuda or source.dtype != torch.int32 or source.numel() < cap:
        raise ValueError("source must be an int32 device tensor with a slot per output row")
    p = GsDensifyParams(float(prune_weight), float(tau), float(new_log_scale), float(new_weight_logit), int(max_new))
    n_out = ctypes.c_int64(0)
    st = load_library().gs_densify(ctypes.byref(params_in.c()), int(n_in), weight.data_ptr(), ctypes.byref(domain),
                                   ctypes.byref(q), value.data_ptr(), influence.data_ptr(), target.data_ptr(),
                                   _ptr(defined), ctypes.byref(p), ctypes.byref(params_out.c()), cap,
                                   source.data_ptr(), ctypes.byref(n_out), work.data_ptr(),
                                   work.numel() * work.element_size(), _stream(stream))
    if st == GS_ERR_CAPACITY:
        raise GsError(st, load_library().gs_last_error().decode(errors="replace") + f" (kept {n_out.value})")
    _check(st)
    return int(n_out.value)


def backward_pair_count(index: Index, query: Query, plan: Optional[torch.Tensor], work: torch.Tensor,
                        stream=None) -> int:
    """(Gaussian, query) pairs gs_sample_backward tests, for measurement
    (waits for the count; overwrites work)."""
    q = query.c()
    out = ctypes.c_int64(0)
    st = load_library().gs_backward_pair_count(ctypes.byref(index.c), ctypes.byref(q), _ptr(plan),
                                               0 if plan is None else plan.numel(), work.data_ptr(), work.numel(),
                                               ctypes.byref(out), _stream(stream))
    _check(st)
    return int(out.value)


def sample_pair_counts(index: Index, query: Query, plan: Optional[torch.Tensor], work: torch.Tensor,
                       stream=None):
    """(tests, contributing): the (Gaussian, query) pairs gs_sample tests and
    those passing the cutoff, for measurement (plan: the one a gs_sample call
    filled; waits for the counts; overwrites work)."""
    q = query.c()
    t, c = ctypes.c_int64(0), ctypes.c_int64(0)
    st = load_library().gs_sample_pair_counts(ctypes.byref(index.c), ctypes.byref(q), _ptr(plan),
                                              0 if plan is None else plan.numel(), work.data_ptr(), work.numel(),
                                              ctypes.byref(t), ctypes.byref(c), _stream(stream))
    _check(st)
    return int(t.value), int(c.value)


def profile_enable(on: bool = True) -> None:
    load_library().gs_profile_enable(1 if on else 0)


def profile_select(name=None) -> None:
    """Record only the kernel `name` (None: every kernel)."""
    load_library().gs_profile_select(None if name is None else name.encode())


def profile_reset() -> None:
    load_library().gs_profile_reset()


def profile_read(max_entries: int = 64):
    """{kernel name: (launches, total milliseconds)} recorded while enabled."""
    L = load_library()
    names = (ctypes.c_char_p * max_entries)()
    counts = (ctypes.c_int64 * max_entries)()
    ms = (ctypes.c_double * max_entries)()
    n = L.gs_profile_read(names, counts, ms, max_entries)
    return {names[i].decode(): (int(counts[i]), float(ms[i])) for i in range(min(n, max_entries))}
