"""Pins of the parity checkers themselves: the forward verdict
(oracle.accept_forward) and the gradient bar (harness.grad_tolerance) must
accept what float32 may legitimately produce and reject plausible mistakes
of a sampler: a relative error a few times the 1e-5 forward target, a
dropped contributing pair, a flipped definedness, a wrong variant at an
ambiguous point, and a 1e-3 error in any one gradient column. The stand-in
"device" results here are the oracle's own float64 values with a planted
mistake; no GPU is used. CPU only."""
import numpy as np
import pytest

import oracle
import synth
from harness import TAU, grad_tolerance, kappa


def scene(seed=3, n=60, npts=3000):
    """Near-isotropic Gaussians (small kappa, so the float32 allowances stay
    far below the planted errors) around the middle of the box."""
    g = synth.random_gaussians(seed, n, log_mu=np.log(0.05), log_sd=0.05, lo=0.3, hi=0.7)
    pts = synth.random_points(seed + 1, npts, 0.25, 0.75)
    return g, pts


def clean(ref):
    """Non-ambiguous defined points whose float32 allowances leave the total
    tolerance below 2.5e-5 relative (1e-5 plus at most 1.5e-5)."""
    amb = oracle.ambiguous_points(ref, TAU)
    d = ref.defined.astype(bool)
    tight = (ref.b_phi + 1e-7 < 1.5e-5 * np.abs(ref.phi)) & (ref.b_inf < 1.5e-5 * ref.inf)
    return d & ~amb & tight


def test_most_points_of_a_workload_hold_a_tight_tolerance():
    """On the first configuration's Gaussians (kappa up to a few) the
    conditioning allowances stay small: at nine points in ten a 3e-5
    relative error in Phi exceeds the tolerance."""
    w = synth.WORKLOADS["c1_grid32"]
    g = synth.make_gaussians(w)
    pts = oracle.voxel_centers(w.dims, ids=np.arange(0, 32 ** 3, 7, dtype=np.uint32))
    ref = oracle.forward(g, pts)
    d = ref.defined.astype(bool)
    frac = clean(ref)[d].mean()
    assert frac > 0.9, frac


def test_accepts_the_float32_rounding_of_the_reference():
    g, pts = scene()
    ref = oracle.forward(g, pts)
    ok, stats = oracle.accept_forward(ref, ref.phi.astype(np.float32), ref.inf.astype(np.float32))
    assert ok.all() and stats["failed"] == 0
    assert ref.defined.sum() > 1000


@pytest.mark.parametrize("rel", [3e-5, -3e-5])
def test_rejects_a_small_relative_error_in_phi(rel):
    g, pts = scene()
    ref = oracle.forward(g, pts)
    c = clean(ref)
    assert c.sum() > 500
    phi = ref.phi * (1 + rel * c)
    ok, _ = oracle.accept_forward(ref, phi, ref.inf)
    assert not ok[c].any()
    assert ok[~c].all()


def test_rejects_a_small_relative_error_in_i():
    g, pts = scene()
    ref = oracle.forward(g, pts)
    c = clean(ref)
    ok, _ = oracle.accept_forward(ref, ref.phi, ref.inf * (1 + 3e-5 * c))
    assert not ok[c].any()


def test_rejects_a_dropped_contributing_pair():
    """Leave out, at every point, the intersecting Gaussian of largest
    weight there: I and Phi move by far more than the tolerance."""
    g, pts = scene(n=40, npts=1500)
    ref = oracle.forward(g, pts)
    c = clean(ref) & (ref.ncontrib >= 2)
    idx = np.nonzero(c)[0][:200]
    assert len(idx) > 100
    # each Gaussian's own contribution a = w G at the chosen points
    a = np.stack([oracle.forward(g.subset(np.array([i])), pts[idx]).i_base for i in range(g.n)], axis=1)
    rejected = 0
    for j, p in enumerate(idx):
        drop = int(np.argmax(a[j]))
        rest = g.subset(np.array([i for i in range(g.n) if i != drop]))
        r2 = oracle.forward(rest, pts[p:p + 1])
        ok, _ = oracle.accept_forward(oracle_slice(ref, p), [r2.phi[0]], [r2.inf[0]])
        rejected += not ok[0]
    assert rejected == len(idx)


def oracle_slice(ref, p):
    out = oracle.ForwardResult(1)
    for k, v in vars(ref).items():
        setattr(out, k, v[p:p + 1].copy())
    return out


def test_rejects_a_flipped_definedness():
    g, pts = scene()
    ref = oracle.forward(g, pts)
    c = clean(ref)
    phi, inf = ref.phi.copy(), ref.inf.copy()
    phi[c], inf[c] = 0.0, 0.0                    # defined points reported undefined
    ok, _ = oracle.accept_forward(ref, phi, inf)
    assert not ok[c].any()
    und = ~ref.defined.astype(bool) & ~oracle.ambiguous_points(ref, TAU)
    assert und.sum() > 50
    phi, inf = ref.phi.copy(), ref.inf.copy()
    phi[und], inf[und] = 0.5, 0.02               # undefined points reported defined
    ok, _ = oracle.accept_forward(ref, phi, inf)
    assert not ok[und].any()


def synthetic(k, i_base, v_base, a, v, tau=TAU):
    """A one-point oracle result with k ambiguous pairs of weights a and
    values v on top of a non-ambiguous part (i_base, v_base)."""
    r = oracle.ForwardResult(1)
    r.namb[0] = k
    r.i_base[0], r.v_base[0] = i_base, v_base
    kk = min(k, oracle.AMB_KEEP)
    r.amb_a[0, :kk], r.amb_v[0, :kk] = a[:kk], v[:kk]
    r.amb_tot[0] = (sum(a), min(v), max(v))
    I = i_base + sum(a)                          # the float64 reference takes them all in
    r.inf[0] = I
    r.phi[0] = (v_base + sum(x * y for x, y in zip(a, v))) / I
    r.defined[0] = 1
    r.ncontrib[0] = 5 + k
    return r


def test_ambiguous_points_match_one_variant():
    a, v = [0.004, 0.003], [0.9, 0.1]
    r = synthetic(2, 0.5, 0.25, a, v)
    # the pair of weight 0.004 left out (float32 put it past the cutoff)
    I = 0.5 + 0.003
    ok, _ = oracle.accept_forward(r, [(0.25 + 0.003 * 0.1) / I], [I])
    assert ok[0]
    # a value that is no variant: rejected
    ok, _ = oracle.accept_forward(r, [(0.25 + 0.003 * 0.1) / I * (1 + 1e-3)], [I])
    assert not ok[0]
    # no variant drops I below the base
    ok, _ = oracle.accept_forward(r, [0.5], [0.49])
    assert not ok[0]


def test_many_ambiguous_pairs_are_bounded_not_waved_through():
    k = oracle.AMB_KEEP + 3
    a = [0.002] * k
    v = [0.2 + 0.05 * j for j in range(k)]
    r = synthetic(k, 0.4, 0.2, a, v)
    I_mid = 0.4 + 0.002 * 5
    ok, stats = oracle.accept_forward(r, [(0.2 + 0.002 * sum(v[:5])) / I_mid], [I_mid])
    assert ok[0] and stats["ambiguous_bounded"] == 1
    # I outside [base, base + all]: rejected
    ok, _ = oracle.accept_forward(r, [0.5], [0.39])
    assert not ok[0]
    ok, _ = oracle.accept_forward(r, [0.5], [0.4 + 0.002 * k + 0.01])
    assert not ok[0]
    # Phi outside the hull of the base value and the ambiguous values: rejected
    ok, _ = oracle.accept_forward(r, [0.95], [I_mid])
    assert not ok[0]
    # undefined although the base alone is well above tau: rejected
    ok, _ = oracle.accept_forward(r, [0.0], [0.0])
    assert not ok[0]


# --------------------------------------------------------------- gradients

def grad_case(seed=5):
    """Random cotangents on overlapping Gaussians: the sums cancel."""
    g = synth.random_gaussians(seed, 30, log_mu=np.log(0.05), log_sd=0.3, lo=0.35, hi=0.65)
    pts = synth.random_points(seed, 2500, 0.3, 0.7).astype(np.float64)
    gp = synth.random_normal(seed, len(pts)).astype(np.float64)
    gi = synth.random_normal(seed + 7, len(pts)).astype(np.float64)
    ref = oracle.forward(g, pts)
    amb = oracle.ambiguous_points(ref, TAU)
    gp[amb] = 0
    gi[amb] = 0
    grad, ab, K, mab, tab = oracle.backward(g, pts, ref.phi, ref.inf, gp, gi, pairs=True)
    return g, pts, gp, gi, ref, grad, ab, grad_tolerance(grad, ab, kappa(g), K, mab, tab, g.scale, g.rot)


def octant_case(log_sd=0.6):
    """A well-conditioned case: isolated anisotropic Gaussians, each with 30
    points in one octant of its own frame (u_k in [0.2, 1.5]) and the
    cotangents (0.1, 1) everywhere, so no gradient sum cancels much."""
    from scipy.spatial.transform import Rotation
    rng = np.random.default_rng(1)
    n = 20
    centers = np.stack(np.meshgrid(*(np.linspace(0.2, 0.8, 3),) * 3, indexing="ij"), -1).reshape(-1, 3)[:n]
    g = synth.random_gaussians(9, n, log_mu=np.log(0.02), log_sd=log_sd)
    g.mean[:] = centers
    pts = []
    for i in range(n):
        q = g.rot[i].astype(np.float64)
        q /= np.linalg.norm(q)
        R = Rotation.from_quat([q[1], q[2], q[3], q[0]]).as_matrix()
        u = rng.uniform(0.2, 1.5, size=(30, 3))
        pts.append(g.mean[i] + (u * g.scale[i].astype(np.float64)) @ R.T)
    pts = np.concatenate(pts).astype(np.float32).astype(np.float64)
    gp, gi = np.full(len(pts), 0.1), np.ones(len(pts))
    ref = oracle.forward(g, pts)
    assert np.all(ref.ncontrib == 1) and not oracle.ambiguous_points(ref, TAU).any()
    grad, ab, K, mab, tab = oracle.backward(g, pts, ref.phi, ref.inf, gp, gi, pairs=True)
    return g, grad, grad_tolerance(grad, ab, kappa(g), K, mab, tab, g.scale, g.rot)


def test_gradient_bar_accepts_float32_rounding():
    g, pts, gp, gi, ref, grad, ab, tol = grad_case()
    assert np.all(np.abs(grad.astype(np.float32).astype(np.float64) - grad) <= tol)
    g, grad, tol = octant_case()
    assert np.all(np.abs(grad.astype(np.float32).astype(np.float64) - grad) <= tol)


@pytest.mark.parametrize("col", range(12))
def test_gradient_bar_rejects_a_1e3_error_in_any_column(col):
    """A relative error of 1e-3 in one column (dmu x3, ds x3, dq x4, dv,
    dw) fails for most Gaussians of the well-conditioned case, and the
    other columns still pass."""
    g, grad, tol = octant_case()
    bad = grad.copy()
    bad[:, col] *= 1 + 1e-3
    fail = np.abs(bad - grad) > tol
    nz = np.abs(grad[:, col]) > 0
    assert nz.sum() == g.n
    assert fail[:, col].mean() >= 0.6, fail[:, col].mean()
    assert not fail[:, [c for c in range(12) if c != col]].any()


def test_gradient_bar_rejects_a_dropped_pair():
    """The gradients with one contributing (Gaussian, point) pair left out
    of a Gaussian's sum (the pair nearest its mean) are rejected for almost
    every Gaussian, with random cotangents."""
    g, pts, gp, gi, ref, grad, ab, tol = grad_case()
    rejected = 0
    for i in range(g.n):
        sup = np.nonzero(oracle.support(g, pts, np.array([i])))[0]
        keep = np.ones(len(pts), bool)
        d2 = ((pts[sup] - g.mean[i].astype(np.float64)) ** 2).sum(axis=1)
        keep[sup[np.argmin(d2)]] = False         # the pair nearest the mean
        g2, _ = oracle.backward(g, pts, ref.phi, ref.inf, gp * keep, gi * keep, select=np.array([i]))
        rejected += bool((np.abs(g2[0] - grad[i]) > tol[i]).any())
    assert rejected >= 0.9 * g.n, rejected


def test_quaternion_moment_map_against_the_oracle():
    """The map from whitened-frame moments to dL/dq that the quaternion bar
    uses reproduces the oracle's per-pair quaternion gradient: for one
    Gaussian, sum_pairs dL/dQ u u^T pushed through it equals column 6..9."""
    from harness import M2_INDEX, quat_moment_map
    g, pts, gp, gi, ref, grad, ab, tol = grad_case()
    i = 4
    q = g.rot[i].astype(np.float64)
    qh = q / np.linalg.norm(q)
    from harness import rot_of
    R = rot_of(qh)
    s = g.scale[i].astype(np.float64)
    d = pts - g.mean[i].astype(np.float64)
    u = (d @ R) / s
    Q = (u * u).sum(axis=1)
    use = (Q <= 2 * np.log(1 / np.float64(np.float32(TAU)))) & ref.defined.astype(bool)
    a = float(g.weight[i]) * np.exp(-0.5 * Q[use])
    dLda = gp[use] * (float(g.value[i]) - ref.phi[use]) / ref.inf[use] + gi[use]
    c = -0.5 * a * dLda
    m2 = np.array([(c * u[use, m] * u[use, k]).sum() for m, k in M2_INDEX])
    np.testing.assert_allclose(quat_moment_map(g.scale[i], g.rot[i]) @ m2, grad[i, 6:10], rtol=1e-9,
                               atol=1e-12 * np.abs(grad[i, 6:10]).max())


def test_triangular_moment_map_against_the_oracle():
    """The map from triangular-frame moments (c = C d, C the upper Cholesky
    factor of Sigma^-1) to (dL/dmu, dL/ds, dL/dq) that the gradient bar uses
    reproduces the oracle's per-pair gradients of columns 0..9 for several
    Gaussians."""
    from harness import moment_map, rot_of
    g, pts, gp, gi, ref, grad, ab, tol = grad_case()
    T = 2 * np.log(1 / np.float64(np.float32(TAU)))
    checked = 0
    for i in range(g.n):
        q = g.rot[i].astype(np.float64)
        R = rot_of(q / np.linalg.norm(q))
        s = g.scale[i].astype(np.float64)
        M = np.diag(1.0 / s) @ R.T
        C = np.linalg.cholesky(M.T @ M).T
        d = pts - g.mean[i].astype(np.float64)
        c = d @ C.T
        Q = (c * c).sum(axis=1)
        use = (Q <= T) & ref.defined.astype(bool)
        if use.sum() < 5:
            continue
        a = float(g.weight[i]) * np.exp(-0.5 * Q[use])
        dLda = gp[use] * (float(g.value[i]) - ref.phi[use]) / ref.inf[use] + gi[use]
        w = -0.5 * a * dLda
        m = np.concatenate([(w[:, None] * c[use]).sum(axis=0),
                            [(w * c[use, j] * c[use, k]).sum() for j, k in ((0, 0), (0, 1), (0, 2), (1, 1), (1, 2), (2, 2))]])
        np.testing.assert_allclose(moment_map(g.scale[i], g.rot[i]) @ m, grad[i, :10], rtol=1e-9,
                                   atol=1e-12 * np.abs(grad[i, :10]).max())
        checked += 1
    assert checked >= 10
