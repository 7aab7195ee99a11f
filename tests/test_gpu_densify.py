"""Parity of weight pruning and sample-error densification (gs_densify,
Sec. 4.2.1; false negatives first, Sec. 4.2.2) with the oracle, and the
index rebuilt on the new set.

The output count, the source map (which Gaussians are kept, which samples
spawn new ones and in which order) and every copied or set parameter are
bit-exact; a new Gaussian's mean is bit-exact with the oracle's float32
position of its sample; its value logit (float64 on both sides, rounded
once on the device) lies within half a float32 ulp."""
import math

import numpy as np
import pytest

import oracle
import synth
from harness import TAU, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_01164_amd as gs
    gs.load_library()


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def params(n, seed):
    g = np.random.default_rng(seed)
    return (g.random((n, 3)).astype(np.float32), g.normal(-4.8, 0.4, (n, 3)).astype(np.float32),
            g.standard_normal((n, 4)).astype(np.float32), g.standard_normal(n).astype(np.float32),
            g.normal(-3.0, 2.0, n).astype(np.float32))


def weights_of(wl):
    return (1.0 / (1.0 + np.exp(-wl.astype(np.float64)))).astype(np.float32)


def outputs(nq, seed, tau=TAU):
    """Sampler-like (Phi, I), targets and volume flags, with many equal
    errors and false negatives."""
    g = np.random.default_rng(seed)
    phi = g.random(nq).astype(np.float32)
    inf = (tau * (1.0 + 3.0 * g.random(nq))).astype(np.float32)
    undef = g.random(nq) < 0.05
    phi[undef] = 0.0
    inf[undef] = 0.0
    y = g.random(nq).astype(np.float32)
    q = g.random(nq) < 0.3
    phi[q] = np.round(phi[q] * 16) / 16
    y[q] = np.round(y[q] * 16) / 16
    y[g.random(nq) < 0.02] = 0.0
    y[g.random(nq) < 0.02] = 1.0
    d = (g.random(nq) > 0.1).astype(np.uint8)
    return phi, inf, y, d


def run_densify(pin, n_in, w, grid, query, phi, inf, y, d, max_new, cap, tau2=0.005, new_ls=-5.0, new_wl=-4.59512,
                tau=TAU):
    import torch
    import paper_2607_01164_amd as gs
    m, ls, rot, vl, wl = pin
    ps = gs.ParamSet(dev(m), dev(ls), dev(rot), dev(vl), dev(wl))
    out = gs.ParamSet.empty(cap, "cuda")
    for t in (out.mean, out.log_scale, out.rot, out.value_logit, out.weight_logit):
        t.fill_(float("nan"))
    src = torch.full((cap,), -(2 ** 31), dtype=torch.int32, device="cuda")
    work = gs.alloc_densify_work(n_in, query, "cuda")
    n = gs.gs_densify(ps, n_in, dev(w), grid, query, dev(phi), dev(inf), dev(y), None if d is None else dev(d), tau2,
                      tau, new_ls, new_wl, max_new, out, src, work)
    torch.cuda.synchronize()
    return n, out, src.cpu().numpy()


def compare(n, out, src, ref, label):
    log(f"  {label}: n_out {n} (kept {ref.kept}, new {ref.n - ref.kept})")
    assert n == ref.n
    np.testing.assert_array_equal(src[:n], ref.source)
    host = lambda t: t[:n].cpu().numpy()
    np.testing.assert_array_equal(host(out.mean), ref.mean)
    np.testing.assert_array_equal(host(out.log_scale), ref.log_scale)
    np.testing.assert_array_equal(host(out.rot), ref.rot)
    np.testing.assert_array_equal(host(out.weight_logit), ref.weight_logit)
    vl = host(out.value_logit).astype(np.float64)
    kept = ref.kept
    np.testing.assert_array_equal(vl[:kept], ref.value_logit[:kept])
    # new value logits: half an ulp of the float64 logit of the clamped target
    assert np.all(np.abs(vl[kept:] - ref.value_logit[kept:]) <= 2.0 ** -23 * np.abs(ref.value_logit[kept:]))


def test_hand_worked_cases_on_device():
    """The oracle's hand-worked fixture, with its positions given by a voxel
    list (sample 4 lists a voxel past the grid: no position)."""
    import paper_2607_01164_amd as gs
    from test_oracle_densify import golden
    w, s, cases = golden()
    pin = params(len(w), 1)
    dims = (8, 8, 8)
    ids = np.array([3, 77, 500, 12, 8 ** 3 + 4, 200, 64, 65, 511], np.uint32)
    assert np.all((ids < 512) == (s[:, 4] != 0))
    grid = gs.make_grid((4, 4, 4))
    q = gs.Query.voxels(dims, dev(ids.view(np.int32)))
    pos = np.zeros((len(ids), 3), np.float32)
    ok = ids < 512
    pos[ok] = oracle.voxel_centers(dims, ids=ids[ok])
    for max_new, cap, want in cases:
        log(f"case densify fixture max_new={max_new} capacity={cap}")
        args = [x.astype(np.float32) for x in (s[:, 0], s[:, 1], s[:, 2])]
        n, out, src = run_densify(pin, len(w), w, grid, q, *args, s[:, 3].astype(np.uint8), max_new, cap, tau2=0.005,
                                  new_ls=-4.0, new_wl=-4.5, tau=0.0625)
        assert n == len(want) and src[:n].tolist() == want, (src[:n], want)
        ref = oracle.densify(*pin, w, pos, ok.astype(np.uint8), *args, s[:, 3], tau2=0.005, tau=0.0625,
                             new_log_scale=-4.0, new_weight_logit=-4.5, max_new=max_new, capacity=cap)
        compare(n, out, src, ref, "fixture")


@pytest.mark.parametrize("kind", ["grid", "voxels", "points", "jitter", "jitter_ids"])
def test_densify_every_query_kind(kind):
    import paper_2607_01164_amd as gs
    n_in = 5000
    pin = params(n_in, 2)
    w = weights_of(pin[4])
    lo, hi = (-0.5, 0.0, 0.25), (1.5, 1.0, 0.75)
    grid = gs.make_grid((8, 6, 5), lo, hi)
    dims = (24, 20, 10)
    nvox = 24 * 20 * 10
    g = np.random.default_rng(3)
    if kind == "grid":
        q, nq = gs.Query.grid(dims), nvox
        pos, ok = oracle.voxel_centers(dims, lo, hi), np.ones(nvox, np.uint8)
    elif kind == "voxels":
        ids = g.choice(nvox + 100, size=3000, replace=False).astype(np.uint32)
        q, nq = gs.Query.voxels(dims, dev(ids.view(np.int32))), 3000
        ok = (ids < nvox).astype(np.uint8)
        pos = np.zeros((nq, 3), np.float32)
        pos[ok != 0] = oracle.voxel_centers(dims, lo, hi, ids=ids[ok != 0])
    elif kind == "points":
        pts = g.uniform(-0.6, 1.6, (4000, 3)).astype(np.float32)
        q, nq = gs.Query.pts(dev(pts)), 4000
        pos, ok = pts, np.ones(nq, np.uint8)
    elif kind == "jitter":
        u = synth.jitter_offsets(4, nvox)
        q, nq = gs.Query.jitter(dims, dev(u)), nvox
        pos, ok = oracle.jitter_positions(dims, u, lo, hi), np.ones(nvox, np.uint8)
    else:
        ids = g.choice(nvox, size=2500, replace=False).astype(np.uint32)
        ids[:5] = nvox + np.arange(5)
        u = synth.jitter_offsets(5, 2500)
        q, nq = gs.Query.jitter(dims, dev(u), dev(ids.view(np.int32))), 2500
        ok = (ids < nvox).astype(np.uint8)
        pos = np.zeros((nq, 3), np.float32)
        pos[ok != 0] = oracle.jitter_positions(dims, u[ok != 0], lo, hi, ids=ids[ok != 0])
    phi, inf, y, d = outputs(nq, 6)
    kept = int(np.count_nonzero(w >= np.float32(0.005)))
    for max_new, cap, flags in ((700, kept + 400, True), (10 ** 6, n_in + nq, False), (0, kept, True)):
        log(f"case densify {kind} nq={nq} max_new={max_new} capacity={cap} flags={flags}")
        dd = d if flags else None
        n, out, src = run_densify(pin, n_in, w, grid, q, phi, inf, y, dd, max_new, cap)
        ref = oracle.densify(*pin, w, pos, ok, phi, inf, y, dd, tau2=0.005, tau=TAU, new_log_scale=-5.0,
                             new_weight_logit=-4.59512, max_new=max_new, capacity=cap)
        compare(n, out, src, ref, kind)


def test_densify_training_size():
    """The structured training step's size: 262,144 Gaussians (weights
    sigmoid(N(-3, 2)), about 12 % below 0.005), 128^3 jittered samples, up
    to 52,428 new Gaussians (a fifth of the count) within a capacity of
    262,144."""
    import paper_2607_01164_amd as gs
    n_in = 262144
    pin = params(n_in, 7)
    w = weights_of(pin[4])
    dims = (128, 128, 128)
    nq = 128 ** 3
    u = synth.jitter_offsets(1, nq, iteration=3)
    grid = gs.make_grid((36, 36, 36))
    q = gs.Query.jitter(dims, dev(u))
    phi, inf, y, d = outputs(nq, 8)
    log("case densify at the training size")
    n, out, src = run_densify(pin, n_in, w, grid, q, phi, inf, y, None, 52428, n_in)
    pos = oracle.jitter_positions(dims, u)
    ref = oracle.densify(*pin, w, pos, np.ones(nq, np.uint8), phi, inf, y, None, tau2=0.005, tau=TAU,
                         new_log_scale=-5.0, new_weight_logit=-4.59512, max_new=52428, capacity=n_in)
    assert ref.n - ref.kept == min(52428, n_in - ref.kept)
    compare(n, out, src, ref, "training size")


def test_capacity_error_and_empty_inputs():
    import paper_2607_01164_amd as gs
    pin = params(300, 9)
    w = weights_of(pin[4])
    kept = int(np.count_nonzero(w >= np.float32(0.005)))
    grid = gs.make_grid((4, 4, 4))
    pts = np.random.default_rng(10).random((100, 3)).astype(np.float32)
    q = gs.Query.pts(dev(pts))
    phi, inf, y, d = outputs(100, 11)
    log("case densify capacity error")
    with pytest.raises(gs.GsError) as e:
        run_densify(pin, 300, w, grid, q, phi, inf, y, d, 10, kept - 1)
    assert e.value.status == gs.GS_ERR_CAPACITY and f"kept {kept}" in str(e.value)
    log("case densify with no Gaussians")
    empty = tuple(a[:0] for a in pin)
    n, out, src = run_densify(empty, 0, w[:0], grid, q, phi, inf, y, d, 30, 50)
    ref = oracle.densify(*empty, w[:0], pts, np.ones(100, np.uint8), phi, inf, y, d, tau2=0.005, tau=TAU,
                         new_log_scale=-5.0, new_weight_logit=-4.59512, max_new=30, capacity=50)
    compare(n, out, src, ref, "no Gaussians")
    log("case densify with no samples")
    q0 = gs.Query.pts(dev(np.zeros((0, 3), np.float32)))
    e0 = np.zeros(0, np.float32)
    n, out, src = run_densify(pin, 300, w, grid, q0, e0, e0, e0, None, 30, 300)
    assert n == kept and src[:n].tolist() == np.nonzero(w >= np.float32(0.005))[0].tolist()


def test_rebuilt_index_matches_oracle():
    """Densify, activate the new set and rebuild the index: the index of the
    new Gaussians is bit-exact with the oracle's (Sec. 4.1.1, Sec. 4.1.2)."""
    import torch
    import paper_2607_01164_amd as gs
    w_ = synth.WORKLOADS["c1_grid32"]
    ls, vl, wl = synth.raw_params(w_)
    base = synth.make_gaussians(w_)
    wl = wl - 2.5  # push some weights below the pruning threshold
    n_in = w_.n_gauss
    pin = (base.mean, ls, base.rot, vl, wl)
    w = weights_of(wl)
    dims = (32, 32, 32)
    nq = 32 ** 3
    u = synth.jitter_offsets(0, nq, iteration=11)
    grid = gs.make_grid(w_.index_cells)
    q = gs.Query.jitter(dims, dev(u))
    phi, inf, y, d = outputs(nq, 12)
    log("case densify then rebuild the index")
    cap = n_in
    n, out, src = run_densify(pin, n_in, w, grid, q, phi, inf, y, None, 800, cap, new_ls=math.log(0.02))
    kept = int(np.count_nonzero(w >= np.float32(0.005)))
    assert kept < n_in and n == min(n_in, kept + 800)
    sc = torch.empty(n, 3, device="cuda")
    va = torch.empty(n, device="cuda")
    we = torch.empty(n, device="cuda")
    gs.gs_activate(out.raw(n), 0.0, sc, va, we)
    g_new = gs.Gaussians(out.mean[:n], sc, out.rot[:n], va, we)
    idx = gs.build_index(g_new, grid, TAU)
    torch.cuda.synchronize()
    host_g = synth.Gaussians(out.mean[:n].cpu().numpy(), sc.cpu().numpy(), out.rot[:n].cpu().numpy(),
                             va.cpu().numpy(), we.cpu().numpy())
    P = idx.n_pairs
    log(f"  rebuilt index: {n} Gaussians, {P} pairs")
    from harness import check_index_arrays, gpu_boxes
    check_index_arrays(host_g, w_.index_cells, (0, 0, 0), (1, 1, 1), TAU, idx.keys[:P].cpu().numpy().view(np.uint32),
                       idx.gids[:P].cpu().numpy().view(np.uint32), idx.cell_offsets.cpu().numpy().view(np.uint32),
                       gpu_boxes(idx, n), label="rebuilt")
    # the next iteration samples the densified set: forward and backward on
    # new jittered positions, against the oracle
    from harness import Run, check_backward, check_forward, masked_cotangents
    u2 = synth.jitter_offsets(0, nq, iteration=12)
    log("  next iteration on the densified set")
    r = Run(host_g, w_.index_cells, "jitter", dims=dims, offsets=u2)
    phi2, inf2 = r.forward()
    ref2, _ = check_forward(r, phi2, inf2, label="forward after densification")
    gv, gi = synth.random_normal(13, nq), synth.random_normal(14, nq)
    gv, gi, _ = masked_cotangents(ref2, gv, gi)
    grads = r.backward(gv, gi)
    sel = np.random.default_rng(15).choice(n, size=min(n, 400), replace=False)
    sel = np.unique(np.concatenate([sel, np.arange(kept, n)[:200]]))  # new Gaussians among them
    check_backward(r, grads, sel, np.arange(nq), gv, gi, label="backward after densification")
