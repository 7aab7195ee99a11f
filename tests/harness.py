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


def gpu_boxes(index, n: int) -> np.ndarray:
    """The float32 cell boxes the GPU preprocess wrote, read back from the
    index workspace (the library's layout: at its start a 32-byte box per
    Gaussian, (x0, y0, z0, flag) and (x1, y1, z1, 0), empty when x1 < x0),
    as [n, 6] = (x0, y0, z0, x1, y1, z1) with -1 for empty boxes."""
    raw = index.work[0: 32 * n].cpu().numpy().view(np.int32).reshape(n, 8)
    box = np.concatenate([raw[:, 0:3], raw[:, 4:7]], axis=1)
    box[raw[:, 4] < raw[:, 0]] = -1
    return box


def check_index_arrays(g, cells, lo, hi, tau, keys, gids, offs, boxes, reach_sel=None, label=""):
    """The GPU index against the oracle, by the properties the paper fixes
    (Sec. 4.1.1, Sec. 4.1.2):
      * every Gaussian's float32 cell box equals the oracle's, bit for bit;
      * the pairs are in strictly increasing (cell key, Gaussian id) order,
        so no pair repeats, and cell_offsets[k] = #pairs with key < k;
      * each Gaussian lists only cells of its box, and at least every cell
        it reaches (the oracle's exact float64 minimum of Q over the cell is
        within the cutoff), checked for the Gaussians reach_sel (all when
        None)."""
    t0 = time.time()
    cells = tuple(int(c) for c in cells)
    ncells = cells[0] * cells[1] * cells[2]
    rbox, rcnt = oracle.index_boxes(g, cells, lo, hi, tau)
    np.testing.assert_array_equal(boxes, rbox)
    P = len(keys)
    k64, g64 = keys.astype(np.int64), gids.astype(np.int64)
    assert np.all(k64 < ncells) and np.all(g64 < g.n)
    code = k64 * (1 << 32) + g64
    assert np.all(np.diff(code) > 0), "pairs not in strictly increasing (key, gid) order"
    np.testing.assert_array_equal(offs.astype(np.int64), np.searchsorted(k64, np.arange(ncells + 1), side="left"))
    cx, cy, cz = k64 % cells[0], (k64 // cells[0]) % cells[1], k64 // (cells[0] * cells[1])
    b = rbox[g64]
    inside = (b[:, 0] <= cx) & (cx <= b[:, 3]) & (b[:, 1] <= cy) & (cy <= b[:, 4]) & (b[:, 2] <= cz) & (cz <= b[:, 5])
    assert inside.all(), f"{int((~inside).sum())} listed cells outside their Gaussian's box"
    sel = np.arange(g.n) if reach_sel is None else np.asarray(reach_sel, dtype=np.int64)
    rc, rk = oracle.reached_cells(g, cells, select=sel, lo=lo, hi=hi, tau=tau)
    want = np.repeat(sel, rc) * ncells + rk.astype(np.int64)
    have = np.sort(g64 * ncells + k64)
    pos = np.clip(np.searchsorted(have, want), 0, max(P - 1, 0))
    found = (have[pos] == want) if P > 0 else np.zeros(len(want), bool)
    if not found.all():
        miss = np.nonzero(~found)[0][:10]
        for m in miss:
            log(f"    reached but not listed: gaussian {want[m] // ncells} cell {want[m] % ncells}")
    assert found.all(), f"{int((~found).sum())} reached cells not listed"
    log(f"  index {label}: P={P}, box cells {int(rcnt.sum())}, reached by {len(sel)} checked Gaussians "
        f"{int(rc.sum())} (oracle {time.time() - t0:.1f}s)")


def check_index(run: Run, reach_sample=None):
    """check_index_arrays on a Run's index; reach_sample: check the reached
    cells of that many seeded Gaussians (the 64 with the most box cells
    among them) instead of all."""
    keys, gids, offs = run.index_arrays()
    boxes = gpu_boxes(run.index, run.g.n)
    sel = None
    if reach_sample is not None and reach_sample < run.g.n:
        rbox, rcnt = oracle.index_boxes(run.g, run.cells, run.lo, run.hi, run.tau)
        big = np.argsort(-rcnt, kind="stable")[:64]
        rnd = np.random.default_rng(97).choice(run.g.n, size=reach_sample, replace=False)
        sel = np.unique(np.concatenate([big, rnd]))
    check_index_arrays(run.g, run.cells, run.lo, run.hi, run.tau, keys, gids, offs, boxes, sel)


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


def rot_of(q):
    """R(q) for the components (w, x, y, z) taken as they are, Hamilton
    convention (quadratic in q; a unit q gives a rotation)."""
    w, x, y, z = q
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - w * z), 2 * (x * z + w * y)],
                     [2 * (x * y + w * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w * x)],
                     [2 * (x * z - w * y), 2 * (y * z + w * x), 1 - 2 * (x * x + y * y)]])


M2_INDEX = ((0, 0), (0, 1), (0, 2), (1, 1), (1, 2), (2, 2))
OWN_ROUNDING = 2.0 ** -48


def quat_moment_map(scale, rot):
    """[4, 6]: the linear map from a Gaussian's whitened-frame second moments
    m2 = sum dL/dQ u u^T (entries 00 01 02 11 12 22, each off-diagonal one
    standing for both of its places) to dL/dq of the raw quaternion. With
    d = R S u, dL/dR = sum dL/dQ 2 d (u / s)^T = 2 R S m2 S^-1; then
    dL/dqhat_i = sum_jk dL/dR_jk dR_jk/dqhat_i (R is quadratic in qhat, so a
    central difference of step 1 is exact), projected on the tangent of the
    unit sphere and divided by |q|."""
    q = np.asarray(rot, np.float64)
    qn = np.linalg.norm(q)
    qh = q / qn
    s = np.asarray(scale, np.float64)
    R = rot_of(qh)
    dR = np.stack([(rot_of(qh + e) - rot_of(qh - e)) / 2.0 for e in np.eye(4)])  # [4, 3, 3]
    out = np.zeros((4, 6))
    for c, (m, k) in enumerate(M2_INDEX):
        E = np.zeros((3, 3))
        E[m, k] = E[k, m] = 1.0
        G = 2.0 * R @ np.diag(s) @ E @ np.diag(1.0 / s)
        dqh = np.einsum("ijk,jk->i", dR, G)
        out[:, c] = (dqh - qh * (qh @ dqh)) / qn
    return out


def moment_map(scale, rot):
    """[10, 9]: the linear map from a Gaussian's triangular-frame moments
    m1 = sum dL/dQ c and m2 = sum dL/dQ c c^T (entries 00 01 02 11 12 22,
    off-diagonal ones standing for both places), c = C d with C the upper
    Cholesky factor of Sigma^-1 = R S^-2 R^T, to (dL/dmu, dL/ds, dL/dq).
    u = S^-1 R^T d = O c with O = S^-1 R^T C^-1 orthogonal, so the
    whitened-frame moments are O m1 and O m2 O^T; then dL/dmu = -2 R S^-1
    (O m1) = -2 C^T m1, dL/ds_k = -2 (O m2 O^T)_kk / s_k, and dL/dq through
    quat_moment_map."""
    q = np.asarray(rot, np.float64)
    s = np.asarray(scale, np.float64)
    R = rot_of(q / np.linalg.norm(q))
    M = np.diag(1.0 / s) @ R.T
    C = np.linalg.cholesky(M.T @ M).T
    O = M @ np.linalg.inv(C)
    L = quat_moment_map(scale, rot)
    out = np.zeros((10, 9))
    out[0:3, 0:3] = -2.0 * C.T
    for c, (m, k) in enumerate(M2_INDEX):
        E = np.zeros((3, 3))
        E[m, k] = E[k, m] = 1.0
        W = O @ E @ O.T
        out[3:6, 3 + c] = -2.0 * np.diag(W) / s
        out[6:10, 3 + c] = L @ np.array([W[a, b] for a, b in M2_INDEX])
    return out


def grad_tolerance(ref, ab, kap, npairs, mom_abs=None, term_abs=None, scale=None, rot=None, rtol=1e-4):
    """Bar of a float32 gradient against the oracle's float64 one, per
    element: rtol |ref| plus the float32 error of the sum over the
    Gaussian's K pairs, measured against the sizes of what is summed. The
    relative error e of G = exp(-Q/2) (e = eps (9 T kappa + 8), from the
    whitening's 18 eps T kappa in Q) scales a pair's whole term, so it
    costs 2 e of the sum of the absolute per-pair terms (term_abs when
    given, else the sizes A below). The rest is rounding of the sums: the device
    adds each lane's share of the pairs in turn (at most ceil(K / 64) + 1
    additions a lane), then reduces 64 lanes in 6 steps, and each term
    takes a few roundings of its products and of the whitened offset
    (8 eps), so the sums err by at most (ceil(K / 64) + 24) eps of the
    sizes of what they add. For dv and dw those sizes are A (the oracle's
    sums of the per-pair terms at the size of their parts); dL/dmu,
    dL/ds and dL/dq the device forms from moments summed in the frame of
    the triangular factor, so for them the sizes of those moments
    (mom_abs) through the absolute values of the linear map from them
    (moment_map), or A where that is larger."""
    e = EPS32 * (9.0 * T64 * kap + 8.0)
    depth = np.ceil(np.asarray(npairs, dtype=np.float64) / 64.0) + 16.0
    r = ((depth + 8.0) * EPS32)[:, None]
    tol = rtol * np.abs(ref) + (2.0 * e[:, None] + r) * ab
    if mom_abs is not None:
        for i in range(len(ref)):
            if not mom_abs[i].any():
                continue  # no pair (or an invalid Gaussian): the bar above, with A = 0
            J = np.abs(moment_map(scale[i], rot[i]))
            scaled = ab[i, :10] if term_abs is None else term_abs[i]
            tol[i, :10] = (rtol * np.abs(ref[i, :10]) + 2.0 * e[i] * scaled +
                           r[i, 0] * np.maximum(ab[i, :10], J @ mom_abs[i]))
    # the float64 reference's own rounding of its cancelling sums (for a
    # spherical Gaussian dL/dq is exactly zero, the oracle's sum of its
    # per-pair terms a few 1e-18)
    return tol + OWN_ROUNDING * ab


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
    ref, ab, K, mab, tab = oracle.backward(run.g, pts_sup, phi_sup, inf_sup, gv_sup, gi_sup, run.lo, run.hi,
                                           run.tau, select=sel, pairs=True)
    got = grads_gpu[sel]
    tol = grad_tolerance(ref, ab, kappa(run.g)[sel], K, mab, tab, run.g.scale[sel], run.g.rot[sel])
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
