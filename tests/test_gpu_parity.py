"""Parity of the HIP path (through the C-ABI) with the CPU oracle.

Index: bit-exact (keys, Gaussian ids, per-cell ranges). Forward: relative
1e-5 plus the per-point float32 conditioning allowance, with the results
float32 may legitimately produce at points within rounding of the cutoff or
of the definedness threshold accepted. Backward: 1e-4 of (|ref| + the sum of
absolute per-pair terms) plus the conditioning allowance, with cotangents
zeroed at those ambiguous points on both sides.

Small cases compare every output; the five workloads run at full size, in
the launch configuration the benchmark times, and compare sampled outputs
the oracle computes one by one."""
import numpy as np
import pytest

import oracle
import synth
from harness import (TAU, Run, check_backward, check_forward, check_index, check_index_arrays, gpu_boxes, log,
                     masked_cotangents)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_01164_amd as gs
    gs.load_library()


# ---------------------------------------------------------------- small cases

@pytest.mark.parametrize("cells", [(8, 8, 8), (16, 16, 16)])
def test_c1_grid_full(cells):
    w = synth.WORKLOADS["c1_grid32"]
    g = synth.make_gaussians(w)
    log(f"case c1 grid 32^3, cells {cells}")
    r = Run(g, cells, "grid", dims=w.dims)
    check_index(r)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="c1")
    gv, gi = synth.cotangents(w, r.nq)
    gv, gi, amb = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    pts = r.positions()
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="c1 all Gaussians")


@pytest.mark.parametrize("dims,cells", [((24, 20, 12), (8, 4, 3)), ((40, 40, 40), (4, 4, 4)),
                                        ((16, 16, 16), (1, 1, 1)), ((30, 18, 7), (5, 3, 7))])
def test_grid_ragged_cells(dims, cells):
    """Voxels per cell below, above and not a multiple of the wave size,
    a single cell, and non-cubic grids."""
    g = synth.random_gaussians(50, 700, log_mu=np.log(0.04), log_sd=0.5)
    log(f"case grid dims {dims} cells {cells}")
    r = Run(g, cells, "grid", dims=dims)
    check_index(r)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="ragged")
    gv, gi = synth.random_normal(51, r.nq), synth.random_normal(52, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="ragged")


def test_grid_non_unit_box():
    g = synth.random_gaussians(53, 500, log_mu=np.log(0.08), log_sd=0.4, lo=-1.0, hi=2.0)
    lo, hi = (-1.0, -0.5, 0.25), (2.0, 1.5, 1.0)
    log("case non-unit box")
    r = Run(g, (6, 4, 3), "grid", dims=(36, 24, 12), lo=lo, hi=hi)
    check_index(r)
    phi, inf = r.forward()
    check_forward(r, phi, inf, label="box")


def test_voxel_list_small():
    dims = (64, 48, 32)
    nvox = 64 * 48 * 32
    g = synth.random_gaussians(54, 3000, log_mu=np.log(0.03), log_sd=0.5)
    ids = np.random.default_rng(7).choice(nvox, size=20011, replace=False).astype(np.uint32)
    ids[:5] = [nvox, nvox + 17, 0xFFFFFFF0, 0, nvox - 1]  # out-of-range ids are outside the domain
    log("case voxel list 20011 ids")
    r = Run(g, (16, 12, 8), "voxels", dims=dims, ids=ids)
    check_index(r)
    phi, inf = r.forward()
    assert phi[0] == 0 and inf[0] == 0 and phi[1] == 0 and phi[2] == 0
    ok = np.arange(len(ids)) >= 3
    check_forward(r, phi, inf, sel=np.nonzero(ok)[0], label="voxels")
    ref = oracle.forward(g, r.positions(np.nonzero(ok)[0]))
    gv, gi = synth.random_normal(55, r.nq), synth.random_normal(56, r.nq)
    gv[~ok] = 0
    gi[~ok] = 0
    sub = np.nonzero(ok)[0]
    gv, gi, _ = masked_cotangents(ref, gv, gi, where=sub)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), sub, gv[sub], gi[sub], label="voxels")


def test_points_small_with_outside_and_boundary():
    g = synth.random_gaussians(57, 2500, log_mu=np.log(0.04), log_sd=0.6)
    pts = synth.random_points(58, 30000, -0.05, 1.05)
    pts[:6] = [[0, 0, 0], [1, 1, 1], [0, 0.5, 1], [1.0000001, 0.5, 0.5], [-1e-7, 0.5, 0.5], [0.5, 0.5, 0.5]]
    log("case points 30000 incl. outside")
    r = Run(g, (10, 10, 10), "points", points=pts)
    check_index(r)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="points")
    inside = np.all((pts >= 0) & (pts <= 1), axis=1)
    assert np.all(phi[~inside] == 0) and np.all(inf[~inside] == 0)
    gv, gi = synth.random_normal(59, r.nq), synth.random_normal(60, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="points")


def test_backward_with_empty_rows_and_boxes():
    """Points fill only one corner of the domain: many Gaussian boxes hold
    no query, and large Gaussians span several batches of 64 rows, some of
    them empty."""
    g = synth.random_gaussians(71, 1500, log_mu=np.log(0.05), log_sd=0.7)
    pts = synth.random_points(72, 20000, 0.0, 0.45)
    pts[:50] += 0.5
    log("case points in one corner, empty boxes and row batches")
    r = Run(g, (24, 24, 24), "points", points=pts)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="corner")
    gv, gi = synth.random_normal(73, r.nq), synth.random_normal(74, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="corner")


@pytest.mark.parametrize("case", ["one cell", "one pair"])
def test_index_and_backward_without_sort_passes(case):
    """Indexes whose pair sort runs no radix pass: a grid of one cell (every
    key is 0) and an index holding a single pair. The pair ids and the
    emit-to-sorted map the backward reads still come out right."""
    if case == "one cell":
        g = synth.random_gaussians(75, 40, log_mu=np.log(0.08))
        cells = (1, 1, 1)
        pts = synth.random_points(76, 3000)
    else:
        g = synth.random_gaussians(77, 1, log_mu=np.log(0.008), log_sd=0.1)
        g.mean[0] = [0.55, 0.55, 0.55]
        cells = (10, 10, 10)
        pts = g.mean + synth.random_normal(78, 30).reshape(10, 3).astype(np.float32) * 0.005
    log("case sort without passes:", case)
    r = Run(g, cells, "points", points=pts)
    if case == "one pair":
        assert r.index.n_pairs == 1
    check_index(r)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label=case)
    gv, gi = synth.random_normal(79, r.nq), synth.random_normal(80, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label=case)


def test_jitter_queries_full_grid():
    """Training samples (Sec. 4.2.2): one random position per voxel of a
    whole grid, at the caller's offsets."""
    g = synth.random_gaussians(88, 1200, log_mu=np.log(0.05), log_sd=0.5)
    dims = (24, 20, 16)
    n = 24 * 20 * 16
    u = synth.jitter_offsets(88, n)
    log("case jitter, every voxel of 24x20x16")
    r = Run(g, (6, 5, 4), "jitter", dims=dims, offsets=u)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="jitter")
    gv, gi = synth.random_normal(89, n), synth.random_normal(90, n)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="jitter")


def test_jitter_queries_listed_voxels():
    """Jittered positions of listed voxels, with offsets at 0 and just below
    1 and ids past the grid (undefined outputs)."""
    g = synth.random_gaussians(91, 2000, log_mu=np.log(0.04), log_sd=0.5, lo=-0.5, hi=1.5)
    dims = (40, 30, 20)
    nvox = 40 * 30 * 20
    ids = np.random.default_rng(92).choice(nvox, size=9000, replace=False).astype(np.uint32)
    ids[:3] = [nvox, nvox + 5, 0xFFFFFFF0]
    u = synth.jitter_offsets(93, len(ids))
    u[3:20] = 0.0
    u[20:40] = np.nextafter(np.float32(1), np.float32(0))
    lo, hi = (-0.5, -0.25, 0.0), (1.5, 1.25, 1.0)
    log("case jitter, 9000 listed voxels")
    r = Run(g, (8, 6, 5), "jitter", dims=dims, ids=ids, offsets=u, lo=lo, hi=hi)
    phi, inf = r.forward()
    assert np.all(phi[:3] == 0) and np.all(inf[:3] == 0)
    sub = np.arange(3, len(ids))
    check_forward(r, phi, inf, sel=sub, label="jitter listed")
    ref = oracle.forward(g, r.positions(sub), lo, hi)
    gv, gi = synth.random_normal(94, r.nq), synth.random_normal(95, r.nq)
    gv[:3] = 0
    gi[:3] = 0
    gv, gi, _ = masked_cotangents(ref, gv, gi, where=sub)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), sub, gv[sub], gi[sub], label="jitter listed")


def test_points_on_a_fine_index():
    """Point queries on an index of 104^3 cells: more than 2^20 buckets, so
    the work-item offsets scan their group sums in a separate pass."""
    g = synth.random_gaussians(84, 400, log_mu=np.log(0.02), log_sd=0.4)
    pts = synth.random_points(85, 6000)
    log("case points on 104^3 cells")
    r = Run(g, (104, 104, 104), "points", points=pts)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="fine index")
    gv, gi = synth.random_normal(86, r.nq), synth.random_normal(87, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="fine index")


def test_index_tile_spanning_many_empty_gaussians():
    """An emit tile whose Gaussians span more than 2^20 ids (1.1 M Gaussians
    outside the domain, hence without cells, between two groups inside it):
    the emit finds each pair's Gaussian by binary search there."""
    inner = synth.random_gaussians(81, 40, log_mu=np.log(0.1))
    n_out = 1_100_000
    g = synth.random_gaussians(82, 40 + n_out + 40, log_mu=np.log(0.1))
    g.mean[:40] = inner.mean
    g.mean[40:40 + n_out] = 5.0
    log("case emit tile over 1.1 M empty Gaussians")
    r = Run(g, (6, 6, 6), "points", points=synth.random_points(83, 2000))
    check_index(r)
    phi, inf = r.forward()
    check_forward(r, phi, inf, label="wide range")


def test_index_many_row_records_per_tile():
    """Thin needles along the (y, z) diagonal: boxes of more than 64 rows
    (row records) listing a few dozen cells each, so that an emit tile meets
    more such boxes than its task slots and the rest place their own
    records; the index keeps every reached cell, and the forward matches."""
    n = 3000
    rng = np.random.default_rng(95)
    mean = rng.uniform(0.15, 0.85, size=(n, 3))
    scale = np.tile(np.array([0.0005, 0.032, 0.0005]), (n, 1)) * rng.uniform(0.9, 1.1, size=(n, 1))
    # rotation by 45 degrees about x: the long axis along (0, 1, 1)
    h = np.sin(np.pi / 8)
    rot = np.tile(np.array([np.cos(np.pi / 8), h, 0.0, 0.0]), (n, 1))
    f = np.float32
    g = synth.Gaussians(mean.astype(f), scale.astype(f), rot.astype(f), rng.random(n).astype(f),
                        rng.uniform(0.2, 1.0, n).astype(f))
    log("case needles, many row-record boxes per emit tile")
    box, cnt = oracle.index_boxes(g, (64, 64, 64))
    rows = (box[:, 4] - box[:, 1] + 1) * (box[:, 5] - box[:, 2] + 1)
    # a capacity that holds a record for every row of these boxes: the
    # records then never run out and every box is trimmed
    r = Run(g, (64, 64, 64), "points", points=synth.random_points(96, 200000), capacity=int(rows.sum()) + 4096)
    assert (rows > 64).mean() > 0.9, "the needles' boxes should hold more than 64 rows"
    keys, gids, offs = r.index_arrays()
    per_box = np.bincount(gids.astype(np.int64), minlength=n)
    assert per_box.mean() < 32, f"{per_box.mean():.1f} pairs a box: too few boxes per tile"
    check_index(r)
    phi, inf = r.forward()
    check_forward(r, phi, inf, label="needles")


def test_dense_items_of_two_queries_a_lane():
    """Launches with many queries give dense cells' work items two queries a
    lane, smaller ones one (a choice by the launch's query count). A uniform
    cloud of 2^24 points on 16^3 cells takes two a lane; its halves take one,
    and every cell stays dense in both (about 4096 and 2048 queries), so the
    walk visits every query's candidates in the same order: the outputs are
    bit-identical, and a sample matches the oracle."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 1 << 24
    # the library's rule: two a lane from 32 items per wave slot (4 SIMDs a
    # CU, seven waves a SIMD) at one a lane
    big = 32 * cus * 4 * 7 * 64
    if not (n >= big > n // 2):
        pytest.skip(f"{cus} compute units: the rule does not split 2^24 points this way")
    g = synth.random_gaussians(97, 4096, log_mu=np.log(0.02))
    pts = synth.random_points(98, n)
    log(f"case dense items: {g.n} Gaussians, {n} uniform points, cells (16, 16, 16)")
    r = Run(g, (16, 16, 16), "points", points=pts)
    phi, inf = r.forward()
    check_forward(r, phi, inf, sel=np.sort(np.random.default_rng(99).choice(n, 2048, replace=False)),
                  label="two a lane")
    del r
    for h in range(2):
        part = slice(h * (n // 2), (h + 1) * (n // 2))
        rh = Run(g, (16, 16, 16), "points", points=pts[part])
        ph, ih = rh.forward()
        assert np.array_equal(ph.view(np.uint32), phi[part].view(np.uint32)), f"half {h}: values differ"
        assert np.array_equal(ih.view(np.uint32), inf[part].view(np.uint32)), f"half {h}: influence differs"
        del rh


def test_dense_walk_keeps_small_gaussians_in_coarse_cells_exact():
    """The dense walk forms Q' from offsets to the cell's centre, whose
    rounding grows with the cell's size in units of the Gaussian's scale;
    chunks that hold a Gaussian far smaller than the cells (coarse) use
    U (p - mu). Tiny Gaussians (scales 0.0003-0.0006) in cells of 0.125, a
    few wide ones that make every point defined, and points on the tiny
    ones' cutoff surfaces in dense cells: every output within the oracle's
    bar (a cutoff decision outside the float32 band would move Phi by about
    1e-3)."""
    rng = np.random.default_rng(101)
    nt, per = 3000, 60
    mean = rng.uniform(0.1, 0.9, size=(nt, 3))
    scale = 0.0003 * rng.uniform(1.0, 2.0, size=(nt, 3))
    q = rng.standard_normal((nt, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    # points on each tiny Gaussian's cutoff ellipsoid (Mahalanobis radius
    # sqrt(T), within 1e-4 of it)
    T = 2.0 * np.log(1.0 / TAU)
    w_, x, y, z = q.T
    R = np.stack([np.stack([1 - 2 * (y * y + z * z), 2 * (x * y - w_ * z), 2 * (x * z + w_ * y)], -1),
                  np.stack([2 * (x * y + w_ * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w_ * x)], -1),
                  np.stack([2 * (x * z - w_ * y), 2 * (y * z + w_ * x), 1 - 2 * (x * x + y * y)], -1)], 1)
    d = rng.standard_normal((nt, per, 3))
    d /= np.linalg.norm(d, axis=2, keepdims=True)
    d *= np.sqrt(T) * (1.0 + rng.uniform(-1e-4, 1e-4, size=(nt, per, 1)))
    pts = (mean[:, None, :] + np.einsum("nij,npj->npi", R, d * scale[:, None, :])).reshape(-1, 3)
    # wide Gaussians under everything
    nw = 8
    wide_mean = rng.uniform(0.2, 0.8, size=(nw, 3))
    f = np.float32
    g = synth.Gaussians(np.concatenate([mean, wide_mean]).astype(f),
                        np.concatenate([scale, np.full((nw, 3), 0.4)]).astype(f),
                        np.concatenate([q, np.tile([1.0, 0.0, 0.0, 0.0], (nw, 1))]).astype(f),
                        rng.random(nt + nw).astype(f), np.concatenate([rng.uniform(0.5, 1.0, nt), np.ones(nw)]).astype(f))
    log(f"case coarse cells: {nt} tiny and {nw} wide Gaussians, {len(pts)} points on cutoff surfaces, cells (8, 8, 8)")
    r = Run(g, (8, 8, 8), "points", points=pts.astype(f))
    phi, inf = r.forward()
    ref, stats = check_forward(r, phi, inf, label="coarse cells")
    assert stats["defined"] > 0.9 * len(pts)


def clustered_points(seed, n, centers, sd):
    rng = np.random.default_rng(seed)
    c = np.asarray(centers, np.float64)[rng.integers(0, len(centers), n)]
    p = c + rng.normal(0.0, sd, size=(n, 3))
    return np.clip(p, 0.0, 1.0).astype(np.float32)


def test_dense_cells_every_output():
    """Clustered points on a coarse index: cells of hundreds to thousands of
    queries, so every dense cell splits into several work items of up to
    two queries a lane, with uneven last items. Every output and every
    Gaussian's gradient against the oracle."""
    g = synth.random_gaussians(101, 1500, log_mu=np.log(0.03), log_sd=0.5)
    pts = clustered_points(102, 200000, [[0.3, 0.3, 0.3], [0.62, 0.55, 0.4], [0.5, 0.8, 0.7]], 0.05)
    log("case dense cells: 200000 clustered points, 8^3 cells")
    r = Run(g, (8, 8, 8), "points", points=pts)
    check_index(r)
    t, inside = oracle.point_cells(pts, (8, 8, 8))
    c = np.clip(np.floor(t), 0, 7).astype(np.int64)
    per = np.bincount(c[:, 0] + 8 * (c[:, 1] + 8 * c[:, 2]), minlength=512)
    log(f"  queries per cell: max {per.max()}, cells with >= 128: {int((per >= 128).sum())}")
    assert per.max() > 2000 and (per >= 128).sum() > 20
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="dense cells")
    gv, gi = synth.random_normal(103, r.nq), synth.random_normal(104, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="dense cells")


@pytest.mark.parametrize("counts", [(1, 2, 3, 4, 5), (31, 32, 33, 63), (64, 65, 127, 128, 129), (255, 256, 257, 700)])
def test_cells_at_layout_boundaries(counts):
    """Cells holding exactly the query counts where the forward changes
    layout or item split (4, 32, 64 queries; 128 per dense item), each cell
    of a 6^3 index filled with that many random points away from its faces,
    a few more points in cells of their own. Every output against the
    oracle."""
    rng = np.random.default_rng(sum(counts))
    g = synth.random_gaussians(105, 900, log_mu=np.log(0.05), log_sd=0.4)
    cells = []
    pts = []
    for k, n in enumerate(counts):
        cx, cy, cz = (k * 2) % 6, (k * 3 + 1) % 6, (k + 2) % 6
        lo = np.array([cx, cy, cz]) / 6.0
        pts.append(lo + (0.02 + 0.96 * rng.random((n, 3))) / 6.0)
        cells.append((cx, cy, cz))
    # a few more points in the x = y = 5 column, which no counted cell uses
    pts.append(np.array([5.0, 5.0, 0.0]) / 6.0 + rng.random((40, 3)) * np.array([1 / 6, 1 / 6, 1.0]))
    pts = np.concatenate(pts).astype(np.float32)
    rng.shuffle(pts)
    log(f"case layout boundaries {counts}: {len(pts)} points")
    r = Run(g, (6, 6, 6), "points", points=pts)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label=f"boundaries {counts}")
    gv, gi = synth.random_normal(106, r.nq), synth.random_normal(107, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="boundaries")


def test_sparse_cells_every_output():
    """Few queries spread over a fine index: almost every occupied cell
    holds one to three queries (lanes are then the cell's candidates)."""
    g = synth.random_gaussians(108, 3000, log_mu=np.log(0.02), log_sd=0.5)
    pts = synth.random_points(109, 4000)
    log("case sparse cells: 4000 points, 32^3 cells")
    r = Run(g, (32, 32, 32), "points", points=pts)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="sparse cells")
    gv, gi = synth.random_normal(110, r.nq), synth.random_normal(111, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="sparse cells")


def test_point_plan_order_matches_oracle():
    """The query ordering kept in the plan (the role of the paper's sample
    BVH, Sec. 5.1.1): a stable sort of the queries by 4 cell + quarter of the
    cell along x (outside points last). Checked by its properties: the order
    is a permutation, keys never decrease, ids ascend within a key, the
    per-key offsets are the ranges, and every query's key is the one a
    float64 recomputation of its cell coordinates gives (within float32
    rounding of a cell or quarter face, either side is accepted)."""
    g = synth.random_gaussians(61, 100)
    pts = synth.random_points(62, 50000, -0.1, 1.1)
    pts[:200] = np.float32(1.0)                 # on the closed box's upper faces
    pts[200:400, 0] = np.float32(0.0)
    cells = (7, 9, 11)
    log("case plan order")
    r = Run(g, cells, "points", points=pts)
    r.forward()
    n = len(pts)
    ncells = 7 * 9 * 11
    plan = r.plan.cpu().numpy()
    keys = plan[: 4 * n].view(np.uint32).astype(np.int64)
    order = plan[_align(4 * n): _align(4 * n) + 4 * n].view(np.uint32).astype(np.int64)
    poff = plan[4 * _align(4 * n): 4 * _align(4 * n) + 4 * (4 * ncells + 2)].view(np.uint32).astype(np.int64)
    np.testing.assert_array_equal(np.sort(order), np.arange(n))
    assert np.all(np.diff(keys) >= 0)
    same = np.diff(keys) == 0
    assert np.all(np.diff(order)[same] > 0), "ids not ascending within a key"
    np.testing.assert_array_equal(poff, np.searchsorted(keys, np.arange(4 * ncells + 2), side="left"))
    kq = np.empty(n, np.int64)
    kq[order] = keys
    t, inside = oracle.point_cells(pts, cells)
    C = np.array(cells, np.float64)
    tol = 2.0 ** -18 * np.maximum(1.0, C)

    def key_of(tt):
        c = np.clip(np.floor(tt), 0, C - 1)
        qx = np.clip(np.floor(4 * (tt[:, 0] - c[:, 0])), 0, 3)
        return 4 * (c[:, 0] + C[0] * (c[:, 1] + C[1] * c[:, 2])) + qx
    ok = np.zeros(n, bool)
    for sx in (-1, 0, 1):
        for sy in (-1, 0, 1):
            for sz in (-1, 0, 1):
                ok |= key_of(t + tol * np.array([sx, sy, sz])).astype(np.int64) == kq
    ok[~inside] = kq[~inside] == 4 * ncells
    exact = key_of(t).astype(np.int64) == kq
    log(f"  {int(exact[inside].sum())} of {int(inside.sum())} inside keys match float64 exactly, "
        f"{int((~inside).sum())} outside")
    assert ok.all(), np.nonzero(~ok)[0][:10]
    assert exact[inside].mean() > 0.999


def _align(x):
    return (x + 255) // 256 * 256


def test_invalid_and_degenerate_gaussians():
    g = synth.random_gaussians(63, 400, log_mu=np.log(0.06))
    g.rot[0] = 0                       # zero quaternion
    g.mean[1, 1] = np.nan
    g.scale[2, 0] = 0
    g.scale[3, 2] = -0.1
    g.value[4] = np.inf
    g.weight[5] = np.nan
    g.mean[6] = [5, 5, 5]              # entirely outside the domain
    g.rot[7] = [1e-30, 0, 0, 0]        # float32 squared norm underflows to zero
    g.rot[8] = [3, -2, 7, 1]           # unnormalised, valid
    log("case invalid Gaussians")
    r = Run(g, (8, 8, 8), "grid", dims=(32, 32, 32))
    check_index(r)
    phi, inf = r.forward()
    assert np.all(np.isfinite(phi)) and np.all(np.isfinite(inf))
    ref, _ = check_forward(r, phi, inf, label="invalid")
    gv, gi = synth.random_normal(64, r.nq), synth.random_normal(65, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    assert np.all(grads[:8] == 0)
    assert np.all(np.isfinite(grads))
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="invalid")


def test_empty_inputs():
    import torch
    import paper_2607_01164_amd as gs
    log("case empty inputs")
    # no Gaussians: every point undefined, nothing to differentiate
    g0 = synth.random_gaussians(66, 1)
    g0 = g0.subset(np.arange(0))
    r = Run(g0, (4, 4, 4), "points", points=synth.random_points(67, 1000))
    assert r.index.n_pairs == 0
    phi, inf = r.forward()
    assert np.all(phi == 0) and np.all(inf == 0)
    # no queries
    g = synth.random_gaussians(68, 50)
    r2 = Run(g, (4, 4, 4), "points", points=np.zeros((0, 3), np.float32))
    assert r2.nq == 0
    r2.forward()
    grads = r2.backward(np.zeros(0, np.float32), np.zeros(0, np.float32))
    assert np.all(grads == 0)
    # a single Gaussian and a single point
    g1 = synth.random_gaussians(69, 1, log_mu=np.log(0.1))
    p1 = g1.mean.copy()
    r3 = Run(g1, (3, 3, 3), "points", points=p1)
    phi, inf = r3.forward()
    assert inf[0] == pytest.approx(float(g1.weight[0]), rel=1e-6)
    assert phi[0] == pytest.approx(float(g1.value[0]), rel=1e-6)
    grads = r3.backward(np.ones(1, np.float32), np.ones(1, np.float32))
    assert grads[0, 10] == pytest.approx(1.0, rel=1e-6)     # dv = gPhi
    assert grads[0, 11] == pytest.approx(1.0, rel=1e-6)     # dw = gI G, G = 1 at the mean
    assert np.all(np.abs(grads[0, :3]) < 1e-3)              # at the mean dmu = 0
    del torch, gs


def test_capacity_error_reports_pairs():
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(70, 300, log_mu=np.log(0.05))
    log("case capacity error")
    dg = __import__("harness").dev_gauss(g)
    grid = gs.make_grid((8, 8, 8))
    P = gs.build_index(dg, grid, TAU).n_pairs
    _, cnt = oracle.index_boxes(g, (8, 8, 8))
    assert 0 < P <= int(cnt.sum())
    idx = gs.Index(grid, g.n, P - 1, "cuda")
    with pytest.raises(gs.GsError) as e:
        gs.gs_build_index(dg, grid, TAU, idx)
    assert e.value.status == gs.GS_ERR_CAPACITY
    assert idx.n_pairs == P
    idx2 = gs.Index(grid, g.n, P, "cuda")
    assert gs.gs_build_index(dg, grid, TAU, idx2) == P
    check_index_arrays(g, (8, 8, 8), (0, 0, 0), (1, 1, 1), TAU, idx2.keys[:P].cpu().numpy().view(np.uint32),
                       idx2.gids[:P].cpu().numpy().view(np.uint32), idx2.cell_offsets.cpu().numpy().view(np.uint32),
                       gpu_boxes(idx2, g.n))


def test_forward_is_deterministic():
    w = synth.WORKLOADS["c1_grid32"]
    g = synth.make_gaussians(w)
    pts = synth.random_points(71, 100000)
    log("case determinism")
    r = Run(g, (8, 8, 8), "points", points=pts)
    a = r.forward()
    b = r.forward()
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    rg = Run(g, (8, 8, 8), "grid", dims=(32, 32, 32))
    c = rg.forward()
    d = rg.forward()
    np.testing.assert_array_equal(c[0], d[0])


def test_planned_sampling_on_a_side_stream_matches_gs_sample():
    """gs_plan_queries on a second stream (over a zeroed plan), while the
    index is rebuilt on the first, then gs_sample_planned and the backward
    (which reads the plan) on the first: outputs and gradients equal the
    one-call path's bit for bit, for points, voxel lists and jittered
    queries (and a grid query needs no plan)."""
    import torch
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(81, 6000, log_mu=np.log(0.02), log_sd=0.5)
    D = (64, 64, 64)
    rng_ids = np.random.default_rng(82).choice(64 ** 3, size=50000, replace=False).astype(np.uint32)
    cases = [("points", dict(points=synth.random_points(83, 90000))),
             ("voxels", dict(dims=D, ids=rng_ids)),
             ("jitter", dict(dims=D, ids=rng_ids, offsets=synth.jitter_offsets(84, len(rng_ids))))]
    for kind, kw in cases:
        log(f"case planned sampling, {kind}")
        r = Run(g, (16, 16, 16), kind, **kw)
        a = r.forward()
        gv, gi = synth.random_normal(85, r.nq), synth.random_normal(86, r.nq)
        ga = r.backward(gv, gi)
        side = torch.cuda.Stream()
        r.plan.zero_()
        torch.cuda.synchronize()
        planned = torch.cuda.Event()
        with torch.cuda.stream(side):
            gs.gs_plan_queries(r.query, r.grid, r.plan, stream=side)
            planned.record(side)
        gs.gs_build_index(r.dg, r.grid, r.tau, r.index)
        torch.cuda.current_stream().wait_event(planned)
        gs.gs_sample_planned(r.dg, r.index, r.query, r.value, r.influence, r.plan)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(r.value[:r.nq].cpu().numpy(), a[0])
        np.testing.assert_array_equal(r.influence[:r.nq].cpu().numpy(), a[1])
        np.testing.assert_array_equal(r.backward(gv, gi), ga)
    rg = Run(g, (16, 16, 16), "grid", dims=D)
    c = rg.forward()
    gs.gs_plan_queries(rg.query, rg.grid, None)
    gs.gs_sample_planned(rg.dg, rg.index, rg.query, rg.value, rg.influence, None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(rg.value.cpu().numpy(), c[0])
    np.testing.assert_array_equal(rg.influence.cpu().numpy(), c[1])


def test_backward_is_deterministic():
    """Every per-Gaussian sum is formed by one wavefront in a fixed order,
    without atomics: repeated backward passes (and a whole repeated step,
    index included) give the same bits, for both packings of Gaussians per
    wave."""
    for n_gauss, seed in ((3000, 73), (70000, 74)):
        g = synth.random_gaussians(seed, n_gauss, log_mu=np.log(0.02), log_sd=0.4)
        pts = synth.random_points(seed + 1, 60000)
        log(f"case backward determinism, {n_gauss} Gaussians")
        r = Run(g, (16, 16, 16), "points", points=pts)
        r.forward()
        gv, gi = synth.random_normal(seed + 2, r.nq), synth.random_normal(seed + 3, r.nq)
        a = r.backward(gv, gi)
        b = r.backward(gv, gi)
        np.testing.assert_array_equal(a, b)
        r2 = Run(g, (16, 16, 16), "points", points=pts)
        r2.forward()
        np.testing.assert_array_equal(r2.backward(gv, gi), a)


def test_sum_rules_hold_on_device():
    """sum_i dv_i = sum over defined points of gPhi, and
    sum_i w_i dw_i = sum over defined points of gI I (any size)."""
    w = synth.WORKLOADS["c1_grid32"]
    g = synth.make_gaussians(w)
    log("case sum rules")
    r = Run(g, (8, 8, 8), "grid", dims=(32, 32, 32))
    phi, inf = r.forward()
    gv, gi = synth.cotangents(w, r.nq, batch_index=5)
    grads = r.backward(gv, gi)
    d = inf > 0
    s1 = float(gv[d].astype(np.float64).sum())
    s2 = float((gi[d].astype(np.float64) * inf[d]).sum())
    assert grads[:, 10].astype(np.float64).sum() == pytest.approx(s1, rel=1e-4, abs=1e-3)
    assert (g.weight.astype(np.float64) * grads[:, 11]).sum() == pytest.approx(s2, rel=1e-4, abs=1e-3)


def test_backward_pair_count():
    """The pairs the backward tests: each row cut to the x-range of the
    cutoff ellipsoid over the row's (y, z) extent, so on a grid (rows of
    voxels) at most the index pairs times the voxels of a cell and at least
    every contributing pair; for points at most the cell lists times the
    cells' queries, and at least every contributing pair (the oracle's
    count), which the cuts of the row ends must never drop."""
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(71, 3000, log_mu=np.log(0.03), log_sd=0.5)
    log("case backward pair count, grid")
    r = Run(g, (8, 8, 8), "grid", dims=(32, 32, 32))
    r.forward()
    work = gs.alloc_backward_work(r.index, r.query, "cuda")
    cnt = gs.backward_pair_count(r.index, r.query, None, work)
    ref = oracle.forward(g, r.positions())
    log(f"  grid: backward tests {cnt}, cell pairs x voxels {r.index.n_pairs * 64}, contributing "
        f"{int(ref.ncontrib.sum())}")
    assert int(ref.ncontrib.sum()) <= cnt <= r.index.n_pairs * 64
    log("case backward pair count, points")
    pts = synth.random_points(72, 40000)
    r = Run(g, (9, 8, 7), "points", points=pts)
    r.forward()
    work = gs.alloc_backward_work(r.index, r.query, "cuda")
    cnt = gs.backward_pair_count(r.index, r.query, r.plan, work)
    tests, contrib = gs.sample_pair_counts(r.index, r.query, r.plan, work)
    keys, gids, offs = r.index_arrays()
    t, inside = oracle.point_cells(pts, (9, 8, 7))
    c = np.clip(np.floor(t), 0, np.array([8, 7, 6])).astype(np.int64)
    per_cell = np.bincount((c[:, 0] + 9 * (c[:, 1] + 8 * c[:, 2]))[inside], minlength=9 * 8 * 7)
    cell_tests = int((np.diff(offs.astype(np.int64)) * per_cell).sum())
    ref = oracle.forward(g, pts)
    ref_contrib = int(ref.ncontrib.sum())
    namb = int(ref.namb.sum())
    log(f"  backward tests {cnt}, forward tests {tests} (cell lists x queries {cell_tests}), contributing {contrib} "
        f"(oracle {ref_contrib}, ambiguous pairs {namb})")
    assert tests == cell_tests
    assert abs(contrib - ref_contrib) <= namb
    assert contrib <= cnt < cell_tests


def test_sample_pair_counts_grid():
    """On a grid every voxel of a cell tests the cell's list; the passing
    pairs are the oracle's contributing pairs up to those within float32
    rounding of the cutoff."""
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(76, 2000, log_mu=np.log(0.03), log_sd=0.5)
    r = Run(g, (8, 8, 8), "grid", dims=(32, 32, 32))
    r.forward()
    work = gs.alloc_backward_work(r.index, r.query, "cuda")
    tests, contrib = gs.sample_pair_counts(r.index, r.query, None, work)
    assert tests == r.index.n_pairs * 64
    ref = oracle.forward(g, r.positions())
    assert abs(contrib - int(ref.ncontrib.sum())) <= int(ref.namb.sum())


def test_backward_quarter_cuts_keep_extreme_points():
    """Points just inside every ellipsoid's x-extremes, d = Sigma e_x
    sqrt(T / Sigma_xx) (1 - 1e-5): the backward cuts a box row to the
    quarters of its end cells that the row's bound reaches, and such points
    sit in those end quarters. Each pair must still be found (the gradients
    against the oracle) and counted."""
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(81, 1500, log_mu=np.log(0.02), log_sd=0.6, lo=0.1, hi=0.9)
    q = g.rot.astype(np.float64)
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    w_, x, y, z = q.T
    R = np.stack([np.stack([1 - 2 * (y * y + z * z), 2 * (x * y - w_ * z), 2 * (x * z + w_ * y)], -1),
                  np.stack([2 * (x * y + w_ * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w_ * x)], -1),
                  np.stack([2 * (x * z - w_ * y), 2 * (y * z + w_ * x), 1 - 2 * (x * x + y * y)], -1)], 1)
    S2 = g.scale.astype(np.float64) ** 2
    Sig = np.einsum("nij,nj,nkj->nik", R, S2, R)
    T = 2.0 * np.log(1.0 / float(np.float32(TAU)))
    d = Sig[:, :, 0] * np.sqrt(T / Sig[:, 0, 0])[:, None] * (1.0 - 1e-5)
    pts = np.concatenate([g.mean + d, g.mean - d]).astype(np.float32)
    log(f"case backward at the ellipsoids' x-extremes, {len(pts)} points")
    r = Run(g, (12, 10, 9), "points", points=pts)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="x-extremes")
    gv, gi = synth.random_normal(82, r.nq), synth.random_normal(83, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label="x-extremes")
    work = gs.alloc_backward_work(r.index, r.query, "cuda")
    assert gs.backward_pair_count(r.index, r.query, r.plan, work) >= int(ref.ncontrib.sum())


@pytest.mark.parametrize("kind", ["points corner", "grid", "jitter"])
def test_backward_four_gaussians_a_wave(kind):
    """From 65,536 Gaussians the backward packs four consecutive Gaussians of
    the spatial order into a wave (fewer take one each): small Gaussians,
    every one of them checked, with empty boxes (points in one corner),
    grid rows and jittered queries."""
    g = synth.random_gaussians(91, 70000, log_mu=np.log(0.012), log_sd=0.4)
    log(f"case backward, four Gaussians a wave: {kind}")
    if kind == "points corner":
        pts = synth.random_points(92, 30000, 0.0, 0.6)
        r = Run(g, (20, 20, 20), "points", points=pts)
    elif kind == "grid":
        r = Run(g, (16, 16, 16), "grid", dims=(48, 48, 48))
    else:
        dims = (40, 36, 32)
        r = Run(g, (20, 18, 16), "jitter", dims=dims, offsets=synth.jitter_offsets(93, 40 * 36 * 32))
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label=kind)
    gv, gi = synth.random_normal(94, r.nq), synth.random_normal(95, r.nq)
    gv, gi, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv, gi)
    check_backward(r, grads, np.arange(g.n), np.arange(r.nq), gv, gi, label=kind)
