"""Shared helpers of the GPU parity tests: run the HIP path through the
C-ABI binding and judge its outputs against the CPU oracle."""
from __future__ import annotations

import math
import sys
import time

import numpy as np

import oracle
import synth

TAU = 0.01
EPS32 = 2.0 ** -24
T64 = 2.0 * math.log(1.0 / float(np.float32(TAU)))


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_gauss(g: synth.Gaussians, device="cuda"):
    import torch
    import paper_2607_01164_amd as gs
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    return gs.Gaussians(t(g.mean), t(g.scale), t(g.rot), t(g.value), t(g.weight))


class Run:
    """One index + forward (+ backward) on the GPU."""

    def __init__(self, g: synth.Gaussians, cells, kind, dims=(0, 0, 0), ids=None, points=None, tau=TAU,
                 lo=(0, 0, 0), hi=(1, 1, 1), capacity=None, offsets=None):
        import torch
        import paper_2607_01164_amd as gs
        self.gs, self.torch = gs, torch
        self.g = g
        self.cells = tuple(cells)
        self.kind = kind
        self.dims = tuple(dims)
        self.lo, self.hi = lo, hi
        self.tau = tau
        self.dg = dev_gauss(g)
        self.grid = gs.make_grid(self.cells, lo, hi)
        self.index = gs.build_index(self.dg, self.grid, tau, capacity=capacity)
        if kind == "grid":
            self.query = gs.Query.grid(dims)
        elif kind == "voxels":
            self.ids_np = np.ascontiguousarray(ids, dtype=np.uint32)
            self.ids_dev = torch.from_numpy(self.ids_np.view(np.int32)).cuda()
            self.query = gs.Query.voxels(dims, self.ids_dev)
        elif kind == "jitter":
            self.ids_np = None if ids is None else np.ascontiguousarray(ids, dtype=np.uint32)
            self.ids_dev = None if ids is None else torch.from_numpy(self.ids_np.view(np.int32)).cuda()
            self.u_np = np.ascontiguousarray(offsets, dtype=np.float32)
            self.u_dev = torch.from_numpy(self.u_np).cuda()
            self.query = gs.Query.jitter(dims, self.u_dev, self.ids_dev)
        else:
            self.points_np = np.ascontiguousarray(points, dtype=np.float32)
            self.points_dev = torch.from_numpy(self.points_np).cuda()
            self.query = gs.Query.pts(self.points_dev)
        self.nq = self.query.size()
        self.plan = gs.alloc_plan(self.query, self.grid, "cuda") if kind != "grid" else None

    def forward(self):
        torch = self.torch
        self.value = torch.empty(max(self.nq, 1), dtype=torch.float32, device="cuda")
        self.influence = torch.empty(max(self.nq, 1), dtype=torch.float32, device="cuda")
        self.gs.gs_sample(self.dg, self.index, self.query, self.value, self.influence, self.plan)
        torch.cuda.synchronize()
        self.phi_np = self.value[:self.nq].cpu().numpy()
        self.inf_np = self.influence[:self.nq].cpu().numpy()
        return self.phi_np, self.inf_np

    def forward_gm(self):
        """The Gaussian-major forward variant; leaves the plan as forward()."""
        torch = self.torch
        self.value = torch.empty(max(self.nq, 1), dtype=torch.float32, device="cuda")
        self.influence = torch.empty(max(self.nq, 1), dtype=torch.float32, device="cuda")
        work = self.gs.alloc_gaussian_major_work(self.query, "cuda")
        self.gs.gs_sample_gaussian_major(self.dg, self.index, self.query, self.value, self.influence, self.plan, work)
        torch.cuda.synchronize()
        self.phi_np = self.value[:self.nq].cpu().numpy()
        self.inf_np = self.influence[:self.nq].cpu().numpy()
        return self.phi_np, self.inf_np

    def backward(self, gv: np.ndarray, gi: np.ndarray):
        torch = self.torch
        self.gv = torch.from_numpy(np.ascontiguousarray(gv, dtype=np.float32)).cuda()
        self.gi = torch.from_numpy(np.ascontiguousarray(gi, dtype=np.float32)).cuda()
        work = self.gs.alloc_backward_work(self.index, self.query, "cuda")
        grads = self.gs.Grads.empty(self.g.n, "cuda")
        self.gs.gs_sample_backward(self.dg, self.index, self.query, self.plan, self.value, self.influence, self.gv,
                                   self.gi, grads, work)
        torch.cuda.synchronize()
        return np.concatenate([grads.mean.cpu().numpy(), grads.scale.cpu().numpy(), grads.rot.cpu().numpy(),
                               grads.value.cpu().numpy()[:, None], grads.weight.cpu().numpy()[:, None]], axis=1)

    def index_arrays(self):
        P = self.index.n_pairs
        keys = self.index.keys[:P].cpu().numpy().view(np.uint32)
        gids = self.index.gids[:P].cpu().numpy().view(np.uint32)
        offs = self.index.cell_offsets.cpu().numpy().view(np.uint32)
        return keys, gids, offs

    def positions(self, sel=None):
        """Canonical float32 positions of the queries (all, or a subset)."""
        if self.kind == "grid":
            ids = None if sel is None else np.asarray(sel, dtype=np.uint32)
            return oracle.voxel_centers(self.dims, self.lo, self.hi, ids=ids)
        if self.kind == "voxels":
            ids = self.ids_np if sel is None else self.ids_np[sel]
            return oracle.voxel_centers(self.dims, self.lo, self.hi, ids=ids)
        if self.kind == "jitter":
            u = self.u_np if sel is None else self.u_np[sel]
            ids = self.ids_np
            if ids is None and sel is not None:
                ids = np.asarray(sel, dtype=np.uint32)
            elif ids is not None and sel is not None:
                ids = ids[sel]
            return oracle.jitter_positions(self.dims, u, self.lo, self.hi, ids=ids)
        return self.points_np if sel is None else self.points_np[sel]


def check_index(run: Run):
    keys, gids, offs = run.index_arrays()
    t0 = time.time()
    rk, rg, ro = oracle.index(run.g, run.cells, run.lo, run.hi, run.tau)
    log(f"  index: P={len(rk)} (oracle {time.time() - t0:.1f}s)")
    assert len(keys) == len(rk), (len(keys), len(rk))
    np.testing.assert_array_equal(offs, ro)
    np.testing.assert_array_equal(keys, rk)
    np.testing.assert_array_equal(gids, rg)


def check_forward(run: Run, phi, inf, sel=None, label=""):
    pts = run.positions(sel)
    t0 = time.time()
    ref = oracle.forward(run.g, pts, run.lo, run.hi, run.tau)
    p = phi if sel is None else phi[sel]
    i = inf if sel is None else inf[sel]
    ok, stats = oracle.accept_forward(ref, p, i, run.tau)
    log(f"  forward {label}: {stats} (oracle {time.time() - t0:.1f}s)")
    if not ok.all():
        bad = np.nonzero(~ok)[0][:10]
        for b in bad:
            log(f"    point {b}: gpu ({p[b]!r}, {i[b]!r}) oracle ({ref.phi[b]!r}, {ref.inf[b]!r}) "
                f"defined={ref.defined[b]} namb={ref.namb[b]} K={ref.ncontrib[b]}")
    assert ok.all(), stats
    return ref, stats


def masked_cotangents(ref, gv, gi, where=None):
    """Cotangents with the points that lie within float32 rounding of a
    cutoff or of the definedness threshold zeroed (on both sides of a
    backward comparison): there the intersecting set itself may differ."""
    amb = oracle.ambiguous_points(ref, TAU)
    gv = gv.copy()
    gi = gi.copy()
    if where is None:
        gv[amb] = 0
        gi[amb] = 0
    else:
        gv[where[amb]] = 0
        gi[where[amb]] = 0
    return gv, gi, amb


def kappa(g: synth.Gaussians) -> np.ndarray:
    """Axis ratio per Gaussian (1 for invalid ones, which contribute nothing)."""
    s = g.scale.astype(np.float64)
    ok = np.all(np.isfinite(s) & (s > 0), axis=1)
    k = np.ones(len(s))
    k[ok] = s[ok].max(axis=1) / s[ok].min(axis=1)
    return k


def grad_tolerance(ref, ab, kap, rtol=1e-4):
    e = EPS32 * (9.0 * T64 * kap + 8.0)
    return rtol * (np.abs(ref) + ab) + 2.0 * e[:, None] * ab


def check_backward(run: Run, grads_gpu: np.ndarray, sel, sup, gv_sup, gi_sup, label=""):
    """grads_gpu: [n, 12] for all Gaussians; the oracle recomputes the
    selected Gaussians from the support queries sup (indices into the
    query). The backward takes the forward's outputs as inputs (Sec. 4.1.4:
    it consumes V, I and their cotangents), so the oracle is evaluated at
    the outputs the GPU forward produced (run.forward() first): near the
    definedness threshold dL/da = gPhi (v - Phi) / I + gI cancels, and the
    forward's own tolerance on Phi would otherwise show up amplified."""
    t0 = time.time()
    sup = np.asarray(sup)
    pts_sup = run.positions(sup)
    phi_sup = run.phi_np[sup].astype(np.float64)
    inf_sup = run.inf_np[sup].astype(np.float64)
    ref, ab = oracle.backward(run.g, pts_sup, phi_sup, inf_sup, gv_sup, gi_sup, run.lo, run.hi, run.tau, select=sel)
    got = grads_gpu[sel]
    tol = grad_tolerance(ref, ab, kappa(run.g)[sel])
    err = np.abs(got - ref)
    ok = err <= tol
    worst = float(np.max(err / np.maximum(tol, 1e-300)))
    log(f"  backward {label}: {len(sel)} Gaussians, max err/tol {worst:.3g}, nonzero ref "
        f"{int((ref != 0).sum())} (oracle {time.time() - t0:.1f}s)")
    if not ok.all():
        r, c = np.nonzero(~ok)
        for a, b in list(zip(r, c))[:10]:
            log(f"    gaussian {sel[a]} col {b}: gpu {got[a, b]!r} oracle {ref[a, b]!r} abs {ab[a, b]!r} "
                f"tol {tol[a, b]!r}")
    assert ok.all()
