"""Pins of the oracle's canonical cell index (Sec. 4.1.1: AABB of the cutoff
ellipsoid on a grid of cells; Sec. 4.1.2: Gaussian-cell pairs ordered by
cell, per-cell ranges) and of the query ordering. CPU only."""
import math

import numpy as np

import synth

TAU = 0.01
RCI64 = math.sqrt(2 * math.log(100.0)) * (1 + 2.0 ** -10)


def sigma_diag(g):
    from scipy.spatial.transform import Rotation
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    s2 = g.scale.astype(np.float64) ** 2
    return np.einsum("njk,nk->nj", R ** 2, s2)


def test_axis_aligned_boxes_closed_form(orc):
    """q = identity: the box half-extent is r_c' s_j on each axis, and the
    row spans are exact: the slab bound's centre line is flat and its
    half-width is r_c' s_x sqrt(1 - d2) with d2 the squared scaled distance
    from the mean to the row's (y, z) rectangle."""
    m = np.array([[0.5, 0.5, 0.5], [0.1, 0.9, 0.33], [0.0, 1.0, 0.5], [0.97, 0.02, 0.5], [0.31, 0.62, 0.47]],
                 np.float32)
    s = np.array([[0.05, 0.02, 0.1], [0.01, 0.01, 0.01], [0.2, 0.05, 0.003], [0.04, 0.04, 0.04],
                  [0.03, 0.045, 0.02]], np.float32)
    n = len(m)
    g = synth.Gaussians(m, s, np.tile(np.float32([1, 0, 0, 0]), (n, 1)), np.full(n, 0.5, np.float32),
                        np.full(n, 0.5, np.float32))
    cells = 16
    box, cnt, trimmed, spans = orc.index_boxes(g, (cells,) * 3, spans=True)
    for i in range(n):
        for j in range(3):
            lo = float(m[i, j]) - RCI64 * float(s[i, j])
            hi = float(m[i, j]) + RCI64 * float(s[i, j])
            assert box[i, j] == max(0, math.floor(lo * cells))
            assert box[i, 3 + j] == min(cells - 1, math.floor(hi * cells))
        nx, ny, nz = box[i, 3:] - box[i, :3] + 1
        assert trimmed[i] == (ny * nz <= 64 and nx <= 16)
        if not trimmed[i]:
            assert cnt[i] == nx * ny * nz
            continue
        total = 0
        for r in range(ny * nz):
            cy, cz = box[i, 1] + r % ny, box[i, 2] + r // ny
            dy = max(cy / cells - m[i, 1], 0.0, m[i, 1] - (cy + 1) / cells) / s[i, 1]
            dz = max(cz / cells - m[i, 2], 0.0, m[i, 2] - (cz + 1) / cells) / s[i, 2]
            d2 = (dy * dy + dz * dz) / RCI64 ** 2
            code = spans[i, r]
            if d2 > 1.0 + 1e-12:
                assert code == 0x0F
                continue
            half = RCI64 * float(s[i, 0]) * math.sqrt(max(0.0, 1.0 - d2))
            xl = min(max(math.floor((float(m[i, 0]) - half) * cells), box[i, 0]), box[i, 3])
            xh = max(min(math.floor((float(m[i, 0]) + half) * cells), box[i, 3]), box[i, 0])
            assert (box[i, 0] + (code & 15), box[i, 0] + (code >> 4)) == (xl, xh), (i, r)
            total += xh - xl + 1
        assert cnt[i] == total


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


def listed_pairs(box, trimmed, spans, cells):
    """(key, gid) of every cell a box lists: all cells of an untrimmed box,
    the row spans of a trimmed one."""
    pairs = []
    C = cells
    for i, b in enumerate(box):
        if b[0] < 0:
            continue
        ny = b[4] - b[1] + 1
        for z in range(b[2], b[5] + 1):
            for y in range(b[1], b[4] + 1):
                x0, x1 = b[0], b[3]
                if trimmed[i]:
                    code = spans[i, (y - b[1]) + ny * (z - b[2])]
                    x0, x1 = b[0] + (code & 15), b[0] + (code >> 4)
                for x in range(x0, x1 + 1):
                    pairs.append((x + C * (y + C * z), i))
    return sorted(pairs)


def test_index_structure_and_order(orc):
    g = synth.random_gaussians(42, 400, log_mu=np.log(0.04), log_sd=0.5)
    cells = 12
    keys, gids, offs = orc.index(g, (cells,) * 3)
    box, cnt, trimmed, spans = orc.index_boxes(g, (cells,) * 3, spans=True)
    P = len(keys)
    assert P == cnt.sum() and offs[-1] == P and offs[0] == 0
    assert trimmed.sum() > 300
    exp = listed_pairs(box, trimmed, spans, cells)
    np.testing.assert_array_equal(keys, [k for k, _ in exp])
    np.testing.assert_array_equal(gids, [i for _, i in exp])
    assert np.all(np.diff(offs.astype(np.int64)) >= 0)
    np.testing.assert_array_equal(offs, np.searchsorted(keys, np.arange(cells ** 3 + 1), side="left"))
    for k in range(cells ** 3):
        seg = gids[offs[k]:offs[k + 1]]
        assert np.all(np.diff(seg.astype(np.int64)) > 0)


def test_index_is_complete_near_the_cutoff(orc):
    """Every point whose exact Q is at most T (1 + 2^-9) lies in a cell of
    the Gaussian's box: points are placed on and just outside the cutoff
    ellipsoid and their cell is looked up in the pair list."""
    from scipy.spatial.transform import Rotation
    g = synth.random_gaussians(43, 300, log_mu=np.log(0.03), log_sd=0.9, lo=0.1, hi=0.9)
    cells = 32
    keys, gids, offs = orc.index(g, (cells,) * 3)
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    rc = math.sqrt(2 * math.log(100.0))
    rng = np.random.default_rng(5)
    lists = {k: set(gids[offs[k]:offs[k + 1]].tolist()) for k in range(cells ** 3) if offs[k + 1] > offs[k]}
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


def test_row_spans_are_tight(orc):
    """The spans keep every cell the (enlarged) cutoff ellipsoid reaches and
    few others: against the exact cell set, found by minimising Q over each
    cell of the box, on C2-like Gaussians."""
    from scipy.optimize import minimize
    from scipy.spatial.transform import Rotation
    g = synth.random_gaussians(45, 150, log_mu=np.log(0.008), log_sd=0.4, lo=0.1, hi=0.9)
    cells = 40
    box, cnt, trimmed, spans = orc.index_boxes(g, (cells,) * 3, spans=True)
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    Tq = RCI64 ** 2
    kept = exact = aabb = 0
    for i in range(g.n):
        if not trimmed[i]:
            continue
        A = np.linalg.inv(R[i] @ np.diag(g.scale[i].astype(np.float64) ** 2) @ R[i].T)
        mu = g.mean[i].astype(np.float64)
        b = box[i]
        ny = b[4] - b[1] + 1
        for cz in range(b[2], b[5] + 1):
            for cy in range(b[1], b[4] + 1):
                code = spans[i, (cy - b[1]) + ny * (cz - b[2])]
                x0, x1 = b[0] + (code & 15), b[0] + (code >> 4)
                for cx in range(b[0], b[3] + 1):
                    aabb += 1
                    lo = np.array([cx, cy, cz]) / cells
                    hi = lo + 1.0 / cells
                    res = minimize(lambda p: (p - mu) @ A @ (p - mu), np.clip(mu, lo, hi),
                                   jac=lambda p: 2 * A @ (p - mu), bounds=list(zip(lo, hi)), method="L-BFGS-B")
                    reach = res.fun <= Tq * (1 - 1e-6)
                    listed = x0 <= cx <= x1
                    exact += reach
                    kept += listed
                    assert listed or not reach, (i, cx, cy, cz, res.fun / Tq)
    print(f"row spans: kept {kept}, exact {exact}, box {aabb}")
    assert kept <= 1.15 * exact and kept < 0.85 * aabb, (kept, exact, aabb)


def test_index_capacity_and_empty(orc):
    g = synth.Gaussians(np.array([[2.0, 2.0, 2.0]], np.float32), np.array([[0.01] * 3], np.float32),
                        np.array([[1, 0, 0, 0]], np.float32), np.array([0.5], np.float32),
                        np.array([0.5], np.float32))
    keys, gids, offs = orc.index(g, (4, 4, 4))
    assert len(keys) == 0 and np.all(offs == 0)


def test_point_order(orc):
    pts = synth.random_points(44, 5000, -0.1, 1.1)
    cells = (8, 4, 16)
    keys, order, offs = orc.point_order(pts, cells)
    ncells = 8 * 4 * 16
    assert sorted(order.tolist()) == list(range(5000))
    assert np.all(np.diff(keys.astype(np.int64)) >= 0)
    for k in np.unique(keys):
        seg = order[keys == k]
        assert np.all(np.diff(seg.astype(np.int64)) > 0)
    np.testing.assert_array_equal(offs, np.searchsorted(keys, np.arange(4 * ncells + 2), side="left"))
    inside = np.all((pts >= 0) & (pts <= 1), axis=1)
    kp = np.empty(5000, np.int64)
    kp[order] = keys
    assert np.all(kp[~inside] == 4 * ncells)
    # cells per axis are powers of two, so t = p * cells is exact and float64
    # reproduces both the cell and the quarter of the cell along x
    t = pts[inside].astype(np.float64) * np.array(cells)
    c = np.clip(np.floor(t), 0, np.array(cells) - 1).astype(np.int64)
    qx = np.clip(np.floor(4 * (t[:, 0] - c[:, 0])), 0, 3).astype(np.int64)
    np.testing.assert_array_equal(kp[inside], 4 * (c[:, 0] + 8 * (c[:, 1] + 4 * c[:, 2])) + qx)


def test_voxel_cells_by_integer_division(orc):
    """Voxel centres fall in cell (voxel // (dims/cells)) on every axis."""
    dims, cells = (32, 16, 64), (8, 4, 16)
    ids = np.random.default_rng(1).choice(32 * 16 * 64, size=3000, replace=False).astype(np.uint32)
    pts = orc.voxel_centers(dims, ids=ids)
    keys, order, offs = orc.point_order(pts, cells)
    kp = np.empty(3000, np.int64)
    kp[order] = keys
    x, y, z = ids % 32, (ids // 32) % 16, ids // (32 * 16)
    # four voxels per cell along x: the quarter is the voxel's place in its cell
    np.testing.assert_array_equal(kp, 4 * (x // 4 + 8 * (y // 4 + 4 * (z // 4))) + x % 4)
