"""Parity of the training epilogue (include/gs_train.h, through the C-ABI)
with the CPU oracle: the activations of Sec. 4.2 and their backward, the
L1 / false-negative (Eq. 4) / false-positive (Eq. 5) losses with their
cotangents, and a structured training step chained through the sampler.

Activations are float64 on both sides and rounded once on the device: each
output lies within half a float32 ulp of the oracle's value (plus the
float64 rounding of the parts where they cancel). Loss counts and
cotangents are bit-exact; the float64 loss sums differ only by summation
order, bounded by 2 n 2^-53 of the sum (every term is non-negative)."""
import math

import numpy as np
import pytest

import oracle
import synth
from harness import TAU, Run, check_backward, check_forward, log, masked_cotangents

pytestmark = pytest.mark.gpu

HALF_ULP = 2.0 ** -24
MIN_SUB = 2.0 ** -149


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_01164_amd as gs
    gs.load_library()


def dev(a, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    return (t if dtype is None else t.to(dtype)).cuda()


def host(t):
    return t.cpu().numpy()


def check_f32(got, ref, extra=0.0, label=""):
    got = np.asarray(got, dtype=np.float64)
    tol = HALF_ULP * np.abs(ref) * (1.0 + 1e-6) + MIN_SUB + extra
    err = np.abs(got - ref)
    worst = float(np.max(err / tol)) if err.size else 0.0
    log(f"  {label}: {err.size} values, max err/tol {worst:.3g}")
    if not np.all(err <= tol):
        i = np.unravel_index(np.argmax(err / tol), err.shape)
        log(f"    worst at {i}: gpu {got[i]!r} oracle {ref[i]!r} tol {tol[i]!r}")
    assert np.all(err <= tol)


def raw_case(n, seed, cap):
    """C2-like free parameters with edge rows: capped norms from far below
    to far above the cap (both sides of the small-norm limit), extreme
    scales, and sigmoid arguments in both tails."""
    w = synth.WORKLOADS["c2_grid256_batch"]
    ls, vl, wl = synth.raw_params(w, n)
    ls, vl, wl = ls.copy(), vl.copy(), wl.copy()
    c = cap if cap > 0 and math.isfinite(cap) else 0.02
    d = np.array([0.48, 0.6, 0.64])  # unit direction
    edges = [1e-6, 5e-5, 9.9e-5, 1e-4, 1.01e-4, 2e-4, 5e-3, 1e-2, 0.5, 1.0, 3.0, 20.0, 1e3]
    rows = [np.log(d * c * t) for t in edges] + [np.array([-200.0, -3.0, -7.0]), np.array([2.0, 1.0, -1.0])]
    logits = [0.0, 1e-8, -1e-8, 17.0, -17.0, 40.0, -40.0, 100.0, -100.0, 88.0, -88.0, 3.5, -0.25, 6.0, -9.0]
    k = min(n, len(rows))
    for i in range(k):
        ls[i] = rows[i]
        vl[i] = logits[i % len(logits)]
        wl[i] = -logits[(i + 3) % len(logits)]
    return ls, vl, wl


@pytest.mark.parametrize("cap", [0.0, 0.02, 0.04, float("inf")])
@pytest.mark.parametrize("n", [1, 15, 1037, 262144])
def test_activate_parity(n, cap):
    import torch
    import paper_2607_01164_amd as gs
    ls, vl, wl = raw_case(n, 1, cap)
    log(f"case activate n={n} cap={cap}")
    raw = gs.RawParams(dev(ls), dev(vl), dev(wl))
    s = torch.empty(n, 3, device="cuda")
    v = torch.empty(n, device="cuda")
    w = torch.empty(n, device="cuda")
    gs.gs_activate(raw, cap, s, v, w)
    torch.cuda.synchronize()
    ocap = float(np.float32(cap)) if math.isfinite(cap) else 0.0  # the library takes the cap as float32
    rs, rv, rw = oracle.activate(oracle.RawGaussians(ls, vl, wl), ocap)
    check_f32(host(s), rs, label="scale")
    check_f32(host(v), rv, label="value")
    check_f32(host(w), rw, label="weight")
    # backward on random cotangents
    g = np.random.default_rng(2)
    ds = g.standard_normal((n, 3)).astype(np.float32)
    dv = g.standard_normal(n).astype(np.float32)
    dw = g.standard_normal(n).astype(np.float32)
    grads = gs.Grads(torch.empty(n, 3, device="cuda"), dev(ds), torch.empty(n, 4, device="cuda"), dev(dv), dev(dw))
    out = gs.RawParams(torch.empty(n, 3, device="cuda"), torch.empty(n, device="cuda"),
                       torch.empty(n, device="cuda"))
    gs.gs_activate_backward(raw, cap, grads, out)
    torch.cuda.synchronize()
    a, b, c = oracle.activate_backward(oracle.RawGaussians(ls, vl, wl), ocap, ds, dv, dw)
    # the capped scale's gradient adds two float64 terms that may cancel:
    # allow float64 rounding of their size, (|ds_k| + |ds|) e_k
    e = np.exp(ls.astype(np.float64))
    parts = (np.abs(ds) + np.linalg.norm(ds.astype(np.float64), axis=1, keepdims=True)) * e
    check_f32(host(out.log_scale), a, extra=1e-14 * parts, label="d log_scale")
    check_f32(host(out.value_logit), b, label="d value_logit")
    check_f32(host(out.weight_logit), c, label="d weight_logit")


def test_activate_in_place():
    """Outputs in the buffers of the inputs they replace give the same bits."""
    import torch
    import paper_2607_01164_amd as gs
    n = 5000
    ls, vl, wl = raw_case(n, 3, 0.02)
    log("case activate in place")
    raw = gs.RawParams(dev(ls), dev(vl), dev(wl))
    s, v, w = torch.empty(n, 3, device="cuda"), torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    gs.gs_activate(raw, 0.02, s, v, w)
    g = np.random.default_rng(4)
    ds, dv, dw = (g.standard_normal((n, 3)).astype(np.float32), g.standard_normal(n).astype(np.float32),
                  g.standard_normal(n).astype(np.float32))
    grads = gs.Grads(None, dev(ds), None, dev(dv), dev(dw))
    out = gs.RawParams(torch.empty(n, 3, device="cuda"), torch.empty(n, device="cuda"),
                       torch.empty(n, device="cuda"))
    gs.gs_activate_backward(raw, 0.02, grads, out)
    # in place: backward first (it reads the raw parameters), into the cotangent buffers
    gs.gs_activate_backward(raw, 0.02, grads, gs.RawParams(grads.scale, grads.value, grads.weight))
    ip = gs.RawParams(raw.log_scale.clone(), raw.value_logit.clone(), raw.weight_logit.clone())
    gs.gs_activate(ip, 0.02, ip.log_scale, ip.value_logit, ip.weight_logit)
    torch.cuda.synchronize()
    assert torch.equal(ip.log_scale, s) and torch.equal(ip.value_logit, v) and torch.equal(ip.weight_logit, w)
    assert torch.equal(grads.scale, out.log_scale) and torch.equal(grads.value, out.value_logit)
    assert torch.equal(grads.weight, out.weight_logit)


def loss_case(n, seed, tau=TAU, eps=0.25):
    """Sampler-like outputs: 20 % undefined (0, 0), influences from just
    above tau to 4 tau with values at the thresholds' float32 neighbours,
    some Phi equal to the target, 20 % of the samples outside the volume."""
    g = np.random.default_rng(seed)
    phi = g.random(n).astype(np.float32)
    t32 = np.float32(tau)
    inf = (tau * (1.0 + 3.0 * g.random(n))).astype(np.float32)
    thr = (1.0 + float(np.float32(eps))) * float(t32)
    t_lo = np.float32(thr)
    edge = np.array([t32, np.nextafter(t32, np.float32(1)), np.nextafter(t_lo, np.float32(0)), t_lo,
                     np.nextafter(t_lo, np.float32(1))], dtype=np.float32)
    pick = g.random(n) < 0.05
    inf[pick] = edge[g.integers(0, len(edge), int(pick.sum()))]
    undef = g.random(n) < 0.2
    phi[undef] = 0.0
    inf[undef] = 0.0
    y = synth.targets(seed, n)
    same = g.random(n) < 0.03
    y[same] = phi[same]
    d = (g.random(n) >= 0.2).astype(np.uint8)
    d[d == 1] = g.integers(1, 256, int((d == 1).sum())).astype(np.uint8)  # any non-zero byte means "in the volume"
    return phi, inf, y, d


def run_loss(phi, inf, y, d, tau, eps, lfn, lfp):
    import torch
    import paper_2607_01164_amd as gs
    n = len(phi)
    gv = torch.full((n,), float("nan"), device="cuda")
    gi = torch.full((n,), float("nan"), device="cuda")
    terms = gs.alloc_loss_terms("cuda")
    work = gs.alloc_loss_work(n, "cuda")
    gs.gs_loss(dev(phi), dev(inf), dev(y), None if d is None else dev(d), tau, eps, lfn, lfp, gv, gi, terms, work)
    torch.cuda.synchronize()
    return gs.read_loss_terms(terms), host(gv), host(gi)


def compare_loss(got, gv, gi, ref, n):
    assert (got["n_defined"], got["n_fn"], got["n_fp"], got["n"]) == (ref.n_defined, ref.n_fn, ref.n_fp, n)
    np.testing.assert_array_equal(gv, ref.grad_value)
    np.testing.assert_array_equal(gi, ref.grad_influence)
    bound = (2 * n + 8) * 2.0 ** -53
    for k in ("l1", "fn", "fp", "total"):
        r = getattr(ref, k)
        assert abs(got[k] - r) <= bound * abs(r), (k, got[k], r)
    log(f"  terms {got}")


@pytest.mark.parametrize("n", [0, 1, 7, 2047, 2048, 2049, 100003, 2 ** 21, 2 ** 21 * 2 + 5])
@pytest.mark.parametrize("with_flags", [True, False])
def test_loss_parity(n, with_flags):
    tau, eps, lfn, lfp = TAU, 0.25, 3.0, 0.5
    phi, inf, y, d = loss_case(n, 10 + n % 97, tau, eps)
    if not with_flags:
        d = None
    log(f"case loss n={n} flags={with_flags}")
    got, gv, gi = run_loss(phi, inf, y, d, tau, eps, lfn, lfp)
    ref = oracle.loss(phi, inf, y, d, tau=tau, eps=eps, lambda_fn=lfn, lambda_fp=lfp)
    compare_loss(got, gv, gi, ref, n)


def test_loss_hand_worked_batch_on_device():
    from test_oracle_train import load_golden
    p, terms, counts, rows = load_golden()
    log("case loss, hand-worked batch")
    got, gv, gi = run_loss(rows[:, 0].astype(np.float32), rows[:, 1].astype(np.float32),
                           rows[:, 2].astype(np.float32), rows[:, 3].astype(np.uint8), p["tau"], p["eps"],
                           p["lambda_fn"], p["lambda_fp"])
    assert [got["l1"], got["fn"], got["fp"], got["total"]] == terms
    assert [got["n_defined"], got["n_fn"], got["n_fp"]] == counts
    np.testing.assert_array_equal(gv, rows[:, 4].astype(np.float32))
    np.testing.assert_array_equal(gi, rows[:, 5].astype(np.float32))


def test_loss_is_deterministic():
    phi, inf, y, d = loss_case(3 * 2 ** 20 + 11, 77)
    log("case loss determinism")
    a = run_loss(phi, inf, y, d, TAU, 0.1, 1.0, 1.0)
    b = run_loss(phi, inf, y, d, TAU, 0.1, 1.0, 1.0)
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])


def test_structured_training_step_chain():
    """One structured training step on the device (Sec. 4.2, Sec. 4.2.2):
    activations -> index -> jittered samples of every voxel -> losses ->
    sampler backward -> activation backward. Each stage is judged against
    the oracle at the inputs the device stage received."""
    import torch
    import paper_2607_01164_amd as gs
    w = synth.WORKLOADS["c1_grid32"]
    ls, vl, wl = synth.raw_params(w)
    base = synth.make_gaussians(w)
    cap = float(np.float32(0.04))  # as the library receives it
    n = w.n_gauss
    log("case training step chain, C1 Gaussians, 32^3 jittered samples")
    raw = gs.RawParams(dev(ls), dev(vl), dev(wl))
    s, v, wt = torch.empty(n, 3, device="cuda"), torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    gs.gs_activate(raw, cap, s, v, wt)
    torch.cuda.synchronize()
    rs, rv, rw = oracle.activate(oracle.RawGaussians(ls, vl, wl), cap)
    check_f32(host(s), rs, label="activated scale")
    g_act = synth.Gaussians(base.mean, host(s), base.rot, host(v), host(wt))
    nq = 32 ** 3
    u = synth.jitter_offsets(w.cfg, nq, iteration=7)
    r = Run(g_act, w.index_cells, "jitter", dims=w.dims, offsets=u)
    phi, inf = r.forward()
    ref, _ = check_forward(r, phi, inf, label="jittered forward")
    y = synth.targets(w.cfg, nq, iteration=7)
    got, gv, gi = run_loss(phi, inf, y, None, TAU, 0.5, 2.0, 1.0)
    lref = oracle.loss(phi, inf, y, None, tau=TAU, eps=0.5, lambda_fn=2.0, lambda_fp=1.0)
    compare_loss(got, gv, gi, lref, nq)
    assert lref.n_fn > 0 and np.count_nonzero(gi) > 0
    gv_m, gi_m, _ = masked_cotangents(ref, gv, gi)
    grads = r.backward(gv_m, gi_m)
    check_backward(r, grads, np.arange(n), np.arange(nq), gv_m, gi_m, label="sampler backward")
    # activation backward on the device's own post-activation gradients
    post = gs.Grads(None, dev(grads[:, 3:6]), None, dev(grads[:, 10].copy()), dev(grads[:, 11].copy()))
    out = gs.RawParams(torch.empty(n, 3, device="cuda"), torch.empty(n, device="cuda"),
                       torch.empty(n, device="cuda"))
    gs.gs_activate_backward(raw, cap, post, out)
    torch.cuda.synchronize()
    a, b, c = oracle.activate_backward(oracle.RawGaussians(ls, vl, wl), cap, grads[:, 3:6], grads[:, 10],
                                       grads[:, 11])
    e = np.exp(ls.astype(np.float64))
    ds = grads[:, 3:6].astype(np.float64)
    parts = (np.abs(ds) + np.linalg.norm(ds, axis=1, keepdims=True)) * e
    check_f32(host(out.log_scale), a, extra=1e-14 * parts, label="d log_scale")
    check_f32(host(out.value_logit), b, label="d value_logit")
    check_f32(host(out.weight_logit), c, label="d weight_logit")
