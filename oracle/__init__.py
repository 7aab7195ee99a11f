"""CPU oracle for sampling a weighted 3D-Gaussian scalar field (W-VEG).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg, never by the product library. It is an
independent float64 brute-force implementation (oracle.c) of the paper's
Eq. 2 and Eq. 3 with the cutoff of Sec. 4.1.1 and the definedness rule of
Sec. 4.1.3, their exact derivatives (Sec. 4.1.4), the canonical float32
cell boxes with their block lists (Sec. 4.1.1, Sec. 4.1.2) and the cells each
Gaussian reaches (an exact float64 minimum of Q over every cell); and (train.c) the training steps on
either side of the path: the activations of Sec. 4.2 and the losses of
Sec. 4.2, Eq. 4 and Eq. 5 with their cotangents.

Every function here is pinned by the tests in tests/test_oracle_*.py against
closed forms, invariants, finite differences and brute-force recounts.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

c_i64 = ctypes.c_int64
c_int = ctypes.c_int
c_float = ctypes.c_float
vp = ctypes.c_void_p


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liboracle.so")
        if not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        L.orc_forward.restype = c_int
        L.orc_forward.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, c_float, c_i64, vp, c_int, c_int,
                                  vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_backward.restype = c_int
        L.orc_backward.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, c_float, c_i64, vp, vp, vp, vp, vp, vp,
                                   c_i64, vp, c_int, c_int, vp, vp, vp, vp, vp]
        L.orc_support.restype = c_int
        L.orc_support.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, c_float, c_i64, vp, c_i64, vp, c_int, vp]
        L.orc_voxel_centers.restype = c_int
        L.orc_voxel_centers.argtypes = [vp, vp, vp, c_i64, vp, vp]
        L.orc_jitter_positions.restype = c_int
        L.orc_jitter_positions.argtypes = [vp, vp, vp, c_i64, vp, vp, vp]
        L.orc_index_boxes.restype = c_i64
        L.orc_index_boxes.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, vp, c_float, vp, vp]
        L.orc_reached_cells.restype = c_int
        L.orc_reached_cells.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, vp, c_float, ctypes.c_double, c_i64, vp,
                                        c_int, vp, vp, c_i64]
        L.orc_index.restype = c_int
        L.orc_index.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, vp, vp, c_float, vp, vp, c_i64, vp, vp]
        L.orc_activate.restype = c_int
        L.orc_activate.argtypes = [c_i64, vp, vp, vp, ctypes.c_double, vp, vp, vp]
        L.orc_activate_backward.restype = c_int
        L.orc_activate_backward.argtypes = [c_i64, vp, vp, vp, ctypes.c_double, vp, vp, vp, vp, vp, vp]
        L.orc_loss.restype = c_int
        L.orc_loss.argtypes = [c_i64, vp, vp, vp, vp, c_float, c_float, c_float, c_float, vp, vp, vp, vp]
        L.orc_densify.restype = c_i64
        L.orc_densify.argtypes = [c_i64, vp, vp, vp, vp, vp, vp, c_float, c_i64, vp, vp, vp, vp, vp, vp, c_float,
                                  c_float, c_float, c_i64, c_i64, vp, vp, vp, vp, vp, vp]
        _LIB = L
    return _LIB


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(vp)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _gauss(g):
    """float32 parameter arrays for the canonical index."""
    return (_f32(g.mean).reshape(-1, 3), _f32(g.scale).reshape(-1, 3), _f32(g.rot).reshape(-1, 4),
            _f32(g.value).reshape(-1), _f32(g.weight).reshape(-1))


def _gauss64(g):
    """float64 parameter arrays (exact copies of float32 inputs, or float64
    values for finite-difference probes)."""
    return (_f64(g.mean).reshape(-1, 3), _f64(g.scale).reshape(-1, 3), _f64(g.rot).reshape(-1, 4),
            _f64(g.value).reshape(-1), _f64(g.weight).reshape(-1))


def _box(lo, hi):
    return _f32(np.asarray(lo, dtype=np.float32).reshape(3)), _f32(np.asarray(hi, dtype=np.float32).reshape(3))


def default_threads() -> int:
    v = os.environ.get("OMP_NUM_THREADS")
    if v and v.isdigit() and int(v) > 0:
        return int(v)
    return max(1, os.cpu_count() or 1)


AMB_KEEP = 8  # ambiguous pairs per point whose a and v the forward keeps one by one


class ForwardResult:
    def __init__(self, n):
        self.phi = np.zeros(n)
        self.inf = np.zeros(n)
        self.defined = np.zeros(n, dtype=np.int32)
        self.ncontrib = np.zeros(n, dtype=np.int32)
        self.namb = np.zeros(n, dtype=np.int32)
        self.i_base = np.zeros(n)
        self.v_base = np.zeros(n)
        self.amb_a = np.zeros((n, AMB_KEEP))
        self.amb_v = np.zeros((n, AMB_KEEP))
        self.amb_tot = np.zeros((n, 3))
        self.b_phi = np.zeros(n)
        self.b_inf = np.zeros(n)


def forward(g, points, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01, prune: bool = True,
            threads: int = 0) -> ForwardResult:
    """Eq. 2 at every point by brute force over all Gaussians (float64)."""
    m, s, q, v, w = _gauss64(g)
    pts = _f64(points).reshape(-1, 3)
    lo_, hi_ = _box(lo, hi)
    n = pts.shape[0]
    r = ForwardResult(n)
    rc = lib().orc_forward(m.shape[0], _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), tau, n, _p(pts),
                           int(prune), threads or default_threads(),
                           _p(r.phi), _p(r.inf), _p(r.defined), _p(r.ncontrib), _p(r.namb), _p(r.i_base),
                           _p(r.v_base), _p(r.amb_a), _p(r.amb_v), _p(r.amb_tot), _p(r.b_phi), _p(r.b_inf))
    if rc != 0:
        raise RuntimeError(f"orc_forward failed ({rc})")
    return r


def backward(g, points, phi, inf, g_phi, g_inf, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01,
             zero_mask=None, select=None, prune: bool = True, threads: int = 0, pairs: bool = False):
    """Exact gradients (float64) of L = sum gPhi*Phi + gI*I with respect to
    every parameter of the selected Gaussians (all when select is None).
    Returns (grad, abs_sum), each [nsel, 12] = dmu(3), ds(3), dq(4), dv, dw,
    and with pairs=True also each Gaussian's number of intersecting pairs
    at the defined points [nsel], the magnitudes of its triangular-frame
    moment sums [nsel, 9] and the sums of the absolute exact per-pair terms
    of dmu, ds, dq [nsel, 10] (see orc_backward)."""
    m, s, q, v, w = _gauss64(g)
    pts = _f64(points).reshape(-1, 3)
    n = pts.shape[0]
    lo_, hi_ = _box(lo, hi)
    phi = np.ascontiguousarray(phi, dtype=np.float64)
    inf = np.ascontiguousarray(inf, dtype=np.float64)
    gp = _f64(g_phi)
    gi = _f64(g_inf)
    zm = None if zero_mask is None else np.ascontiguousarray(zero_mask, dtype=np.uint8)
    sel = None if select is None else np.ascontiguousarray(select, dtype=np.int64)
    nsel = m.shape[0] if sel is None else sel.shape[0]
    grad = np.zeros((nsel, 12))
    ab = np.zeros((nsel, 12))
    K = np.zeros(nsel, dtype=np.int64)
    mab = np.zeros((nsel, 9))
    tab = np.zeros((nsel, 10))
    rc = lib().orc_backward(m.shape[0], _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), tau, n, _p(pts),
                            _p(phi), _p(inf), _p(gp), _p(gi), _p(zm), nsel, _p(sel), int(prune),
                            threads or default_threads(), _p(grad), _p(ab), _p(K), _p(mab), _p(tab))
    if rc != 0:
        raise RuntimeError(f"orc_backward failed ({rc})")
    return (grad, ab, K, mab, tab) if pairs else (grad, ab)


def support(g, points, select, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01, threads: int = 0):
    """Mask of points within the cutoff (plus ambiguity band) of any selected Gaussian."""
    m, s, q, v, w = _gauss64(g)
    pts = _f64(points).reshape(-1, 3)
    lo_, hi_ = _box(lo, hi)
    sel = np.ascontiguousarray(select, dtype=np.int64)
    out = np.zeros(pts.shape[0], dtype=np.uint8)
    rc = lib().orc_support(m.shape[0], _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), tau,
                           pts.shape[0], _p(pts), sel.shape[0], _p(sel), threads or default_threads(), _p(out))
    if rc != 0:
        raise RuntimeError(f"orc_support failed ({rc})")
    return out.astype(bool)


def voxel_centers(dims, lo=(0, 0, 0), hi=(1, 1, 1), ids=None) -> np.ndarray:
    """Canonical float32 voxel centres (x fastest ids); all voxels when ids is None."""
    d = np.asarray(dims, dtype=np.int32).reshape(3)
    lo_, hi_ = _box(lo, hi)
    if ids is None:
        n = int(d[0]) * int(d[1]) * int(d[2])
        idp = None
    else:
        ids = np.ascontiguousarray(ids, dtype=np.uint32)
        n = ids.shape[0]
        idp = ids
    out = np.zeros((n, 3), dtype=np.float32)
    rc = lib().orc_voxel_centers(_p(d), _p(lo_), _p(hi_), n, _p(idp), _p(out))
    if rc != 0:
        raise RuntimeError("orc_voxel_centers failed")
    return out


def jitter_positions(dims, u, lo=(0, 0, 0), hi=(1, 1, 1), ids=None) -> np.ndarray:
    """Canonical float32 training positions lo + (i + u) * voxel size (Sec.
    4.2.2): offsets u [n, 3] for the voxels ids (x fastest), or for every
    voxel in order when ids is None."""
    d = np.asarray(dims, dtype=np.int32).reshape(3)
    lo_, hi_ = _box(lo, hi)
    u = np.ascontiguousarray(u, dtype=np.float32).reshape(-1, 3)
    n = u.shape[0]
    idp = None
    if ids is not None:
        ids = np.ascontiguousarray(ids, dtype=np.uint32)
        if ids.shape[0] != n:
            raise ValueError("one offset row per voxel id")
        idp = ids
    elif n != int(d[0]) * int(d[1]) * int(d[2]):
        raise ValueError("without ids there is one offset row per voxel")
    out = np.zeros((n, 3), dtype=np.float32)
    rc = lib().orc_jitter_positions(_p(d), _p(lo_), _p(hi_), n, _p(idp), _p(u), _p(out))
    if rc != 0:
        raise RuntimeError("orc_jitter_positions failed")
    return out


def index_boxes(g, cells, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01):
    """Canonical float32 cell box of every Gaussian's cutoff ellipsoid
    (Sec. 4.1.1): [n, 6] = (x0, y0, z0, x1, y1, z1), inclusive, -1 when
    empty, and its number of cells."""
    m, s, q, v, w = _gauss(g)
    c = np.asarray(cells, dtype=np.int32).reshape(3)
    lo_, hi_ = _box(lo, hi)
    n = m.shape[0]
    box = np.zeros((n, 6), dtype=np.int32)
    cnt = np.zeros(n, dtype=np.int64)
    P = lib().orc_index_boxes(n, _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), _p(c), tau, _p(box), _p(cnt))
    if P < 0:
        raise ValueError("orc_index_boxes: bad arguments")
    return box, cnt


def reached_cells(g, cells, select=None, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01, margin: float = 0.0,
                  threads: int = 0):
    """For the selected Gaussians (all when None): the keys of the index
    cells holding a point within the cutoff Q <= 2 ln(1/tau), each cell
    widened by `margin` cell widths (exact float64 minimum of Q over the
    cell). Returns (counts [nsel], keys concatenated Gaussian after
    Gaussian, ascending within each)."""
    m, s, q, v, w = _gauss(g)
    c = np.asarray(cells, dtype=np.int32).reshape(3)
    lo_, hi_ = _box(lo, hi)
    n = m.shape[0]
    sel = None if select is None else np.ascontiguousarray(select, dtype=np.int64)
    nsel = n if sel is None else sel.shape[0]
    cnt = np.zeros(nsel, dtype=np.int64)
    th = threads or default_threads()
    rc = lib().orc_reached_cells(n, _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), _p(c), tau, float(margin),
                                 nsel, _p(sel), th, _p(cnt), None, 0)
    if rc != 0:
        raise RuntimeError(f"orc_reached_cells failed ({rc})")
    total = int(cnt.sum())
    keys = np.zeros(max(total, 1), dtype=np.uint32)
    rc = lib().orc_reached_cells(n, _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), _p(c), tau, float(margin),
                                 nsel, _p(sel), th, _p(cnt), _p(keys), total)
    if rc != 0:
        raise RuntimeError(f"orc_reached_cells failed ({rc})")
    return cnt, keys[:total]


def index(g, cells, lo=(0, 0, 0), hi=(1, 1, 1), tau: float = 0.01):
    """Canonical index: (keys, gids, cell_offsets) with pairs ordered by (key, gid)."""
    m, s, q, v, w = _gauss(g)
    c = np.asarray(cells, dtype=np.int32).reshape(3)
    lo_, hi_ = _box(lo, hi)
    n = m.shape[0]
    _, cnt = index_boxes(g, cells, lo, hi, tau)
    P = int(cnt.sum())
    keys = np.zeros(max(P, 1), dtype=np.uint32)
    gids = np.zeros(max(P, 1), dtype=np.uint32)
    ncells = int(c[0]) * int(c[1]) * int(c[2])
    offs = np.zeros(ncells + 1, dtype=np.uint32)
    npairs = c_i64(0)
    rc = lib().orc_index(n, _p(m), _p(s), _p(q), _p(v), _p(w), _p(lo_), _p(hi_), _p(c), tau, _p(keys), _p(gids),
                         P, _p(offs), ctypes.byref(npairs))
    if rc != 0:
        raise RuntimeError(f"orc_index failed ({rc})")
    return keys[:P], gids[:P], offs


def point_cells(points, cells, lo=(0, 0, 0), hi=(1, 1, 1)):
    """float64 cell coordinates t_j = (p_j - lo_j) C_j / (hi_j - lo_j) of
    each point (its cell is floor(t) clamped to the grid) and whether it lies
    in the closed domain box."""
    pts = np.asarray(points, dtype=np.float64).reshape(-1, 3)
    lo_ = np.asarray(lo, dtype=np.float32).astype(np.float64)
    hi_ = np.asarray(hi, dtype=np.float32).astype(np.float64)
    c = np.asarray(cells, dtype=np.float64)
    t = (pts - lo_) * (c / (hi_ - lo_))
    inside = np.all((pts >= lo_) & (pts <= hi_), axis=1)
    return t, inside


def accept_forward(ref: ForwardResult, phi_gpu, inf_gpu, tau: float = 0.01, rtol: float = 1e-5,
                   atol_phi: float = 1e-7):
    """Element-wise parity verdict for float32 forward outputs against the
    oracle. At a point that is not ambiguous: |Phi - ref| <= rtol |ref| +
    B_Phi + atol and |I - ref| <= rtol ref + B_I, both sides defined or
    undefined alike. At an ambiguous point (a pair within the float32 band of
    the cutoff, or I within 2^-16 tau of tau) the result must match one of the
    oracle's variants: each of its k ambiguous pairs in or out, and either
    side of the definedness threshold when I is that close to it. With more
    than AMB_KEEP ambiguous pairs (whose terms are not kept one by one) the
    result must lie within the hull of those variants instead: I between the
    sum without and with every ambiguous pair, Phi between the least and the
    largest of Phi without them and their values. Returns (ok_mask, stats)."""
    phi_gpu = np.asarray(phi_gpu, dtype=np.float64)
    inf_gpu = np.asarray(inf_gpu, dtype=np.float64)
    n = ref.phi.shape[0]
    tau64 = float(np.float32(tau))
    band_i = 2.0 ** -16 * tau64

    def close(phi_r, inf_r, defined_r, bphi, binf):
        ok_def = defined_r & (np.abs(phi_gpu - phi_r) <= rtol * np.abs(phi_r) + bphi + atol_phi) & \
            (np.abs(inf_gpu - inf_r) <= rtol * inf_r + binf)
        ok_und = (~defined_r) & (phi_gpu == 0.0) & (inf_gpu == 0.0)
        return ok_def | ok_und

    defined = ref.defined.astype(bool)
    ok = close(ref.phi, ref.inf, defined, ref.b_phi, ref.b_inf)
    near_tau = np.abs(ref.inf - tau64) <= band_i
    amb_pt = (ref.namb > 0) | near_tau
    idx = np.nonzero(amb_pt & ~ok)[0]
    bounded = 0
    for p in idx:
        k = int(ref.namb[p])
        gp, gi = phi_gpu[p], inf_gpu[p]
        bphi, binf = ref.b_phi[p], ref.b_inf[p]
        gdef = not (gp == 0.0 and gi == 0.0)
        if k > AMB_KEEP:
            bounded += 1
            ib, asum = ref.i_base[p], ref.amb_tot[p, 0]
            if not gdef:
                ok[p] = ib <= tau64 + band_i
                continue
            vals = [ref.amb_tot[p, 1], ref.amb_tot[p, 2]] + ([ref.v_base[p] / ib] if ib > 0 else [])
            lo_p, hi_p = min(vals), max(vals)
            tol_p = rtol * max(abs(lo_p), abs(hi_p)) + bphi + atol_phi
            ok[p] = bool(gi > tau64 - band_i and ib * (1 - rtol) - binf <= gi <= (ib + asum) * (1 + rtol) + binf
                         and lo_p - tol_p <= gp <= hi_p + tol_p)
            continue
        bits = ((np.arange(1 << k)[:, None] >> np.arange(k)[None, :]) & 1).astype(np.float64)
        a = ref.amb_a[p, :k]
        I = ref.i_base[p] + bits @ a
        V = ref.v_base[p] + bits @ (a * ref.amb_v[p, :k])
        if gdef:
            ph = np.where(I > 0, V / np.where(I > 0, I, 1.0), 0.0)
            good = (I > tau64 - band_i) & (np.abs(gp - ph) <= rtol * np.abs(ph) + bphi + atol_phi) & \
                (np.abs(gi - I) <= rtol * I + binf)
        else:
            good = I <= tau64 + band_i
        ok[p] = bool(good.any())
    stats = {
        "n": n,
        "defined": int(defined.sum()),
        "ambiguous": int(amb_pt.sum()),
        "ambiguous_bounded": bounded,
        "failed": int((~ok).sum()),
        "used_allowance": int((defined & ok & ((np.abs(phi_gpu - ref.phi) > rtol * np.abs(ref.phi) + atol_phi) |
                                               (np.abs(inf_gpu - ref.inf) > rtol * ref.inf))).sum()),
    }
    return ok, stats


def ambiguous_points(ref: ForwardResult, tau: float = 0.01) -> np.ndarray:
    tau64 = float(np.float32(tau))
    return (ref.namb > 0) | (np.abs(ref.inf - tau64) <= 2.0 ** -16 * tau64)


class RawGaussians:
    """Free parameters before the activations of Sec. 4.2: log-scales
    [n][3], value and weight logits [n] (means and quaternions pass through
    the activations unchanged and are not needed here)."""

    def __init__(self, log_scale, value_logit, weight_logit):
        self.log_scale = _f64(log_scale).reshape(-1, 3)
        self.value_logit = _f64(value_logit).reshape(-1)
        self.weight_logit = _f64(weight_logit).reshape(-1)
        self.n = self.log_scale.shape[0]


def activate(raw: RawGaussians, cap: float):
    """(scale [n][3], value [n], weight [n]) in float64: sigmoid values and
    weights, exp scales with the soft norm cap c (none when c <= 0)."""
    n = raw.n
    s = np.zeros((n, 3))
    v = np.zeros(n)
    w = np.zeros(n)
    rc = lib().orc_activate(n, _p(raw.log_scale), _p(raw.value_logit), _p(raw.weight_logit), float(cap),
                            _p(s), _p(v), _p(w))
    assert rc == 0, rc
    return s, v, w


def activate_backward(raw: RawGaussians, cap: float, d_scale, d_value, d_weight):
    """Gradients of the free parameters (d log-scale [n][3], d value logit,
    d weight logit) from those of the activated ones, in float64."""
    n = raw.n
    ds, dv, dw = _f64(d_scale).reshape(-1, 3), _f64(d_value).reshape(-1), _f64(d_weight).reshape(-1)
    a = np.zeros((n, 3))
    b = np.zeros(n)
    c = np.zeros(n)
    rc = lib().orc_activate_backward(n, _p(raw.log_scale), _p(raw.value_logit), _p(raw.weight_logit), float(cap),
                                     _p(ds), _p(dv), _p(dw), _p(a), _p(b), _p(c))
    assert rc == 0, rc
    return a, b, c


class LossResult:
    def __init__(self, terms, counts, grad_value, grad_influence):
        self.l1, self.fn, self.fp, self.total = (float(x) for x in terms)
        self.n_defined, self.n_fn, self.n_fp = (int(x) for x in counts)
        self.grad_value = grad_value
        self.grad_influence = grad_influence


def loss(value, influence, target, defined=None, tau=0.01, eps=0.1, lambda_fn=1.0, lambda_fp=1.0) -> LossResult:
    """L1 + false-negative (Eq. 4) + false-positive (Eq. 5) losses of a batch
    of sampler outputs against targets, and the cotangents for the sampler's
    backward (float32). defined: per-sample flag of the original volume, or
    None when every sample is defined there."""
    v, i, y = _f32(value).reshape(-1), _f32(influence).reshape(-1), _f32(target).reshape(-1)
    n = v.shape[0]
    assert i.shape[0] == n and y.shape[0] == n
    d = None if defined is None else np.ascontiguousarray(defined, dtype=np.uint8).reshape(-1)
    terms = np.zeros(4)
    counts = np.zeros(3, dtype=np.int64)
    gv = np.zeros(n, dtype=np.float32)
    gi = np.zeros(n, dtype=np.float32)
    rc = lib().orc_loss(n, _p(v), _p(i), _p(y), _p(d), float(tau), float(eps), float(lambda_fn),
                        float(lambda_fp), _p(terms), _p(counts), _p(gv), _p(gi))
    assert rc == 0, rc
    return LossResult(terms, counts, gv, gi)


class DensifyResult:
    def __init__(self, n_out, kept, mean, log_scale, rot, value_logit, weight_logit, source):
        self.n = n_out
        self.kept = kept
        self.mean, self.log_scale, self.rot = mean, log_scale, rot
        self.value_logit, self.weight_logit, self.source = value_logit, weight_logit, source


def densify(mean, log_scale, rot, value_logit, weight_logit, weight, positions, valid, value, influence, target,
            defined=None, tau2=0.005, tau=0.01, new_log_scale=-5.0, new_weight_logit=-4.59511985,
            max_new=0, capacity=None):
    """Weight pruning and sample-error densification (Sec. 4.2.1, false
    negatives first, Sec. 4.2.2) of a set of free Gaussian parameters
    (float32). positions [nq][3] and valid [nq] give each sample's position
    (as the sampler computes it) and whether it has one. Returns a
    DensifyResult, or raises ValueError when the kept Gaussians alone exceed
    the capacity."""
    mean, log_scale, rot = _f32(mean).reshape(-1, 3), _f32(log_scale).reshape(-1, 3), _f32(rot).reshape(-1, 4)
    vl, wl, w = _f32(value_logit).reshape(-1), _f32(weight_logit).reshape(-1), _f32(weight).reshape(-1)
    n_in = mean.shape[0]
    pos = _f32(positions).reshape(-1, 3)
    nq = pos.shape[0]
    ok = np.ascontiguousarray(valid, dtype=np.uint8).reshape(-1)
    v, i, y = _f32(value).reshape(-1), _f32(influence).reshape(-1), _f32(target).reshape(-1)
    d = None if defined is None else np.ascontiguousarray(defined, dtype=np.uint8).reshape(-1)
    cap = n_in + nq if capacity is None else int(capacity)
    om, ols, orot = np.zeros((cap, 3), np.float32), np.zeros((cap, 3), np.float32), np.zeros((cap, 4), np.float32)
    ovl, owl = np.zeros(cap, np.float32), np.zeros(cap, np.float32)
    src = np.zeros(cap, np.int32)
    r = lib().orc_densify(n_in, _p(mean), _p(log_scale), _p(rot), _p(vl), _p(wl), _p(w), float(tau2), nq, _p(pos),
                          _p(ok), _p(v), _p(i), _p(y), _p(d), float(tau), float(new_log_scale),
                          float(new_weight_logit), int(max_new), cap, _p(om), _p(ols), _p(orot), _p(ovl), _p(owl),
                          _p(src))
    if r < 0:
        raise ValueError(f"{-1 - r} kept Gaussians exceed the capacity {cap}")
    kept = int(np.count_nonzero(w >= np.float32(tau2)))
    return DensifyResult(int(r), kept, om[:r], ols[:r], orot[:r], ovl[:r], owl[:r], src[:r])
