"""Pins of the oracle's canonical cell index (Sec. 4.1.1: AABB of the cutoff
ellipsoid on a grid of cells; Sec. 4.1.2: Gaussian-cell pairs ordered by
cell, per-cell ranges), of the cells each Gaussian reaches (an exact
minimum of Q over every cell), and of the query points' cell coordinates.
CPU only."""
import math

import numpy as np
import pytest

import synth

TAU = 0.01
RCI64 = math.sqrt(2 * math.log(100.0)) * (1 + 2.0 ** -10)


def sigma_diag(g):
    from scipy.spatial.transform import Rotation
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    s2 = g.scale.astype(np.float64) ** 2
    return np.einsum("njk,nk->nj", R ** 2, s2)


T64 = 2 * math.log(1.0 / float(np.float32(TAU)))


def axis_aligned(m, s):
    n = len(m)
    return synth.Gaussians(np.asarray(m, np.float32), np.asarray(s, np.float32),
                           np.tile(np.float32([1, 0, 0, 0]), (n, 1)), np.full(n, 0.5, np.float32),
                           np.full(n, 0.5, np.float32))


AXIS_M = np.array([[0.5, 0.5, 0.5], [0.1, 0.9, 0.33], [0.0, 1.0, 0.5], [0.97, 0.02, 0.5], [0.31, 0.62, 0.47]],
                  np.float32)
AXIS_S = np.array([[0.05, 0.02, 0.1], [0.01, 0.01, 0.01], [0.2, 0.05, 0.003], [0.04, 0.04, 0.04],
                   [0.03, 0.045, 0.02]], np.float32)


def test_axis_aligned_boxes_closed_form(orc):
    """q = identity: the box half-extent is r_c' s_j on each axis."""
    m, s = AXIS_M, AXIS_S
    g = axis_aligned(m, s)
    cells = 16
    box, cnt = orc.index_boxes(g, (cells,) * 3)
    for i in range(len(m)):
        for j in range(3):
            lo = float(m[i, j]) - RCI64 * float(s[i, j])
            hi = float(m[i, j]) + RCI64 * float(s[i, j])
            assert box[i, j] == max(0, math.floor(lo * cells))
            assert box[i, 3 + j] == min(cells - 1, math.floor(hi * cells))
        nx, ny, nz = box[i, 3:] - box[i, :3] + 1
        assert cnt[i] == nx * ny * nz


@pytest.mark.parametrize("margin", [0.0, 0.25])
def test_reached_cells_axis_aligned_closed_form(orc, margin):
    """q = identity: Q = sum_j (d_j / s_j)^2 separates by axis, so its
    minimum over a cell is the sum over axes of (distance from mu_j to the
    cell's (widened) interval / s_j)^2, and a cell is reached when that is at
    most T = 2 ln(1/tau)."""
    m, s = AXIS_M, AXIS_S
    g = axis_aligned(m, s)
    cells = 16
    box, _ = orc.index_boxes(g, (cells,) * 3)
    cnt, keys = orc.reached_cells(g, (cells,) * 3, margin=margin)
    start = np.concatenate([[0], np.cumsum(cnt)])
    for i in range(len(m)):
        want = []
        b = box[i]
        for z in range(b[2], b[5] + 1):
            for y in range(b[1], b[4] + 1):
                for x in range(b[0], b[3] + 1):
                    q = 0.0
                    for j, c in enumerate((x, y, z)):
                        lo, hi = (c - margin) / cells, (c + 1 + margin) / cells
                        d = max(lo - float(m[i, j]), 0.0, float(m[i, j]) - hi) / float(s[i, j])
                        q += d * d
                    if q <= T64:
                        want.append(x + cells * (y + cells * z))
        assert keys[start[i]:start[i + 1]].tolist() == want, i
    # an anisotropic Gaussian reaches fewer cells than its box holds
    assert cnt[0] < (box[0, 3:] - box[0, :3] + 1).prod()


def test_rotated_boxes_against_float64_extent(orc):
    """Rotated, anisotropic Gaussians: the box is the cell range of
    mu +- r_c' sqrt(Sigma_jj) (the exact extent of the ellipsoid along j),
    recomputed in float64; only ends within rounding of a cell face may
    differ."""
    g = synth.random_gaussians(41, 3000, log_mu=np.log(0.03), log_sd=0.8, lo=-0.05, hi=1.05)
    for cells in (8, 32, 64):
        box, cnt = orc.index_boxes(g, (cells,) * 3)
        h = RCI64 * np.sqrt(sigma_diag(g))
        mu = g.mean.astype(np.float64)
        tl, th = (mu - h) * cells, (mu + h) * cells
        near = (np.abs(tl - np.round(tl)) < 1e-4) | (np.abs(th - np.round(th)) < 1e-4)
        miss = (np.floor(th) < 0) | (np.floor(tl) > cells - 1)
        elo = np.clip(np.floor(tl), 0, cells - 1)
        ehi = np.clip(np.floor(th), 0, cells - 1)
        emp = miss.any(axis=1)
        ok_rows = ~near.any(axis=1)
        assert ok_rows.sum() > 2500
        assert np.all((box[:, 0] < 0) == emp)
        sel = ok_rows & ~emp
        np.testing.assert_array_equal(box[sel, :3], elo[sel])
        np.testing.assert_array_equal(box[sel, 3:], ehi[sel])
        np.testing.assert_array_equal(cnt[emp], 0)


def test_index_structure_and_order(orc):
    """The block lists hold every cell of every box (Sec. 4.1.2), ordered by
    cell key and, within a cell, by Gaussian id; offsets are the ranges."""
    g = synth.random_gaussians(42, 400, log_mu=np.log(0.04), log_sd=0.5)
    cells = 12
    keys, gids, offs = orc.index(g, (cells,) * 3)
    box, cnt = orc.index_boxes(g, (cells,) * 3)
    P = len(keys)
    assert P == cnt.sum() and offs[-1] == P and offs[0] == 0
    exp = []
    for i, b in enumerate(box):
        if b[0] < 0:
            continue
        for z in range(b[2], b[5] + 1):
            for y in range(b[1], b[4] + 1):
                for x in range(b[0], b[3] + 1):
                    exp.append((x + cells * (y + cells * z), i))
    exp.sort()
    np.testing.assert_array_equal(keys, [k for k, _ in exp])
    np.testing.assert_array_equal(gids, [i for _, i in exp])
    assert np.all(np.diff(offs.astype(np.int64)) >= 0)
    np.testing.assert_array_equal(offs, np.searchsorted(keys, np.arange(cells ** 3 + 1), side="left"))
    for k in range(cells ** 3):
        seg = gids[offs[k]:offs[k + 1]]
        assert np.all(np.diff(seg.astype(np.int64)) > 0)


def test_index_is_complete_near_the_cutoff(orc):
    """Every point whose exact Q is at most T (1 + 2^-9) lies in a cell of
    the Gaussian's box, and every point with Q <= T in a cell the Gaussian
    reaches: points are placed on and just outside the cutoff ellipsoid and
    their cell is looked up in the pair list and in the reached cells."""
    from scipy.spatial.transform import Rotation
    g = synth.random_gaussians(43, 300, log_mu=np.log(0.03), log_sd=0.9, lo=0.1, hi=0.9)
    cells = 32
    keys, gids, offs = orc.index(g, (cells,) * 3)
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    rc = math.sqrt(2 * math.log(100.0))
    rng = np.random.default_rng(5)
    lists = {k: set(gids[offs[k]:offs[k + 1]].tolist()) for k in range(cells ** 3) if offs[k + 1] > offs[k]}
    rcnt, rkeys = orc.reached_cells(g, (cells,) * 3)
    rstart = np.concatenate([[0], np.cumsum(rcnt)])
    for i in range(300):
        dirs = rng.standard_normal((64, 3))
        dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
        rho = rng.uniform(0.9, 1.0 + 2.0 ** -10, size=64)
        pts = g.mean[i].astype(np.float64) + ((dirs * rc * rho[:, None]) * g.scale[i].astype(np.float64)) @ R[i].T
        pts = pts.astype(np.float32)
        inside = np.all((pts >= 0) & (pts <= 1), axis=1)
        for p in pts[inside]:
            c = np.clip(np.floor(p.astype(np.float32) * np.float32(cells)), 0, cells - 1).astype(int)
            k = c[0] + cells * (c[1] + cells * c[2])
            assert i in lists.get(k, ()), (i, p)
        # and the cells holding points inside the exact cutoff are reached
        d = pts[inside].astype(np.float64) - g.mean[i].astype(np.float64)
        u = (d @ R[i]) / g.scale[i].astype(np.float64)
        Q = (u * u).sum(axis=1)
        c = np.clip(np.floor(pts[inside].astype(np.float64) * cells), 0, cells - 1).astype(np.int64)
        k = c[:, 0] + cells * (c[:, 1] + cells * c[:, 2])
        reached = set(rkeys[rstart[i]:rstart[i + 1]].tolist())
        for kk in k[Q <= T64 * (1 - 1e-9)]:
            assert int(kk) in reached, (i, int(kk))


def test_reached_cells_against_numerical_minimisation(orc):
    """Rotated, anisotropic Gaussians: a cell is reached exactly when a
    bound-constrained numerical minimiser (scipy L-BFGS-B, an independent
    method) finds Q <= T over it; cells whose minimum lies within 10^-6 T
    of T are not judged."""
    from scipy.optimize import minimize
    from scipy.spatial.transform import Rotation
    g = synth.random_gaussians(45, 60, log_mu=np.log(0.012), log_sd=0.6, lo=0.1, hi=0.9)
    cells = 40
    box, _ = orc.index_boxes(g, (cells,) * 3)
    cnt, keys = orc.reached_cells(g, (cells,) * 3)
    start = np.concatenate([[0], np.cumsum(cnt)])
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    judged = reached = 0
    for i in range(g.n):
        A = np.linalg.inv(R[i] @ np.diag(g.scale[i].astype(np.float64) ** 2) @ R[i].T)
        mu = g.mean[i].astype(np.float64)
        b = box[i]
        got = set(keys[start[i]:start[i + 1]].tolist())
        for cz in range(b[2], b[5] + 1):
            for cy in range(b[1], b[4] + 1):
                for cx in range(b[0], b[3] + 1):
                    lo = np.array([cx, cy, cz]) / cells
                    hi = lo + 1.0 / cells
                    res = minimize(lambda p: (p - mu) @ A @ (p - mu), np.clip(mu, lo, hi),
                                   jac=lambda p: 2 * A @ (p - mu), bounds=list(zip(lo, hi)), method="L-BFGS-B",
                                   options={"ftol": 1e-15, "gtol": 1e-12})
                    if abs(res.fun - T64) <= 1e-6 * T64:
                        continue
                    judged += 1
                    k = cx + cells * (cy + cells * cz)
                    assert (k in got) == (res.fun < T64), (i, cx, cy, cz, res.fun / T64)
                    reached += k in got
    print(f"reached cells: {reached} of {judged} judged box cells")
    assert 0 < reached < judged


def test_reached_cells_select_and_margin(orc):
    """A selection returns the same cells as the full call for those
    Gaussians; widening the cells never loses one; invalid Gaussians reach
    none."""
    g = synth.random_gaussians(46, 200, log_mu=np.log(0.03), log_sd=0.7)
    g.scale[5, 1] = 0.0
    cells = (9, 7, 11)
    cnt, keys = orc.reached_cells(g, cells)
    start = np.concatenate([[0], np.cumsum(cnt)])
    sel = np.array([3, 5, 17, 150, 3])
    scnt, skeys = orc.reached_cells(g, cells, select=sel)
    sstart = np.concatenate([[0], np.cumsum(scnt)])
    for a, i in enumerate(sel):
        assert skeys[sstart[a]:sstart[a + 1]].tolist() == keys[start[i]:start[i + 1]].tolist()
    assert cnt[5] == 0
    wcnt, wkeys = orc.reached_cells(g, cells, margin=0.1)
    wstart = np.concatenate([[0], np.cumsum(wcnt)])
    assert np.all(wcnt >= cnt) and wcnt.sum() > cnt.sum()
    for i in range(g.n):
        assert set(keys[start[i]:start[i + 1]].tolist()) <= set(wkeys[wstart[i]:wstart[i + 1]].tolist())


def test_index_capacity_and_empty(orc):
    g = synth.Gaussians(np.array([[2.0, 2.0, 2.0]], np.float32), np.array([[0.01] * 3], np.float32),
                        np.array([[1, 0, 0, 0]], np.float32), np.array([0.5], np.float32),
                        np.array([0.5], np.float32))
    keys, gids, offs = orc.index(g, (4, 4, 4))
    assert len(keys) == 0 and np.all(offs == 0)


def test_point_cells(orc):
    """float64 cell coordinates: on power-of-two grids over [0,1]^3 they are
    p * cells exactly; outside points are flagged; voxel centres fall in
    cell voxel // (dims / cells) on every axis."""
    pts = synth.random_points(44, 5000, -0.1, 1.1)
    cells = (8, 4, 16)
    t, inside = orc.point_cells(pts, cells)
    np.testing.assert_array_equal(inside, np.all((pts >= 0) & (pts <= 1), axis=1))
    np.testing.assert_array_equal(t, pts.astype(np.float64) * np.array(cells, np.float64))
    dims = (32, 16, 64)
    ids = np.random.default_rng(1).choice(32 * 16 * 64, size=3000, replace=False).astype(np.uint32)
    vc = orc.voxel_centers(dims, ids=ids)
    t, inside = orc.point_cells(vc, cells)
    assert inside.all()
    c = np.floor(t).astype(np.int64)
    x, y, z = ids % 32, (ids // 32) % 16, ids // (32 * 16)
    np.testing.assert_array_equal(c, np.stack([x // 4, y // 4, z // 4], axis=1))
    # four voxels per cell along x: the quarter of the cell is the voxel's place in it
    np.testing.assert_array_equal(np.floor(4 * (t[:, 0] - c[:, 0])).astype(np.int64), x % 4)
    # a non-unit box
    t2, _ = orc.point_cells(np.array([[-1.0, 0.5, 2.0]], np.float32), (6, 4, 3), lo=(-1, 0, 1), hi=(2, 1, 4))
    np.testing.assert_allclose(t2, [[0.0, 2.0, 1.0]])
