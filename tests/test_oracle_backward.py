"""Pins of the oracle's backward pass (Sec. 4.1.4, through the activations
of Sec. 4.2 only as far as the normalised quaternion): sum rules, a
single-Gaussian closed form, a scaling identity, rotation invariance and
central finite differences of the float64 forward. CPU only."""
import math

import numpy as np
import pytest

import synth
from test_oracle_forward import concat, one

TAU = 0.01


def loss_and_grad(orc, g, pts, gp, gi, **kw):
    r = orc.forward(g, pts, **kw)
    grad, ab = orc.backward(g, pts, r.phi, r.inf, gp, gi, **kw)
    return r, grad, ab


def cluster(seed, n=24, npts=2500):
    g = synth.random_gaussians(seed, n, log_mu=np.log(0.05), log_sd=0.4, lo=0.35, hi=0.65)
    pts = synth.random_points(seed, npts, 0.25, 0.75).astype(np.float64)
    gp = synth.random_normal(seed, npts).astype(np.float64)
    gi = synth.random_normal(seed + 100, npts).astype(np.float64)
    return g, pts, gp, gi


def test_sum_rules(orc):
    """sum_i dL/dv_i = sum_p gPhi(p) and sum_i w_i dL/dw_i = sum_p gI(p) I(p)
    over defined points (the normalised weights a_i / I sum to one)."""
    g, pts, gp, gi = cluster(21)
    r, grad, ab = loss_and_grad(orc, g, pts, gp, gi)
    d = r.defined.astype(bool)
    assert d.sum() > 1000
    assert grad[:, 10].sum() == pytest.approx(gp[d].sum(), rel=1e-10, abs=1e-10)
    assert (g.weight.astype(np.float64) * grad[:, 11]).sum() == pytest.approx((gi * r.inf)[d].sum(), rel=1e-10)


def test_single_gaussian_closed_form(orc):
    """With one Gaussian Phi = v, so dv = gPhi, dw = gI G,
    dmu = gI w G Sigma^-1 d and ds_k = gI w G u_k^2 / s_k."""
    from scipy.spatial.transform import Rotation
    q = np.array([0.3, -0.4, 0.5, 0.7], dtype=np.float32)
    s = np.array([0.05, 0.09, 0.03], dtype=np.float32)
    mu = np.array([0.5, 0.5, 0.5])
    g = one(mu, s, q, 0.6, 0.8)
    R = Rotation.from_quat([q[1], q[2], q[3], q[0]]).as_matrix()
    s64 = s.astype(np.float64)
    for k, off in enumerate([(0.01, 0.02, -0.03), (-0.05, 0.0, 0.04), (0.0, 0.0, 0.0)]):
        p = (mu + np.asarray(off))[None, :]
        gp, gi = np.array([0.7]), np.array([-1.3])
        r, grad, _ = loss_and_grad(orc, g, p, gp, gi)
        assert r.defined[0] == 1
        d = p[0] - mu
        u = (R.T @ d) / s64
        G = math.exp(-0.5 * float(u @ u))
        w = float(np.float32(0.8))
        icov = R @ np.diag(1 / s64 ** 2) @ R.T
        np.testing.assert_allclose(grad[0, 10], 0.7, rtol=1e-12)
        np.testing.assert_allclose(grad[0, 11], -1.3 * G, rtol=1e-12)
        np.testing.assert_allclose(grad[0, 0:3], -1.3 * w * G * (icov @ d), rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(grad[0, 3:6], -1.3 * w * G * u ** 2 / s64, rtol=1e-9, atol=1e-12)


def test_scale_position_identity_single_point(orc):
    """Q is unchanged by scaling d and s together, so for one query point
    sum_k s_k dL/ds_k = (p - mu) . dL/dmu for every Gaussian."""
    g, _, _, _ = cluster(22, n=30)
    p = np.array([[0.5, 0.49, 0.51]])
    r, grad, _ = loss_and_grad(orc, g, p, np.array([1.1]), np.array([0.4]))
    assert r.defined[0] == 1
    lhs = np.sum(g.scale.astype(np.float64) * grad[:, 3:6], axis=1)
    rhs = np.sum((p - g.mean.astype(np.float64)) * grad[:, 0:3], axis=1)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-9, atol=1e-12)
    assert np.count_nonzero(lhs) >= 3


def test_spherical_quaternion_gradient_is_zero(orc):
    g, pts, gp, gi = cluster(23, n=10)
    g.scale[:] = g.scale[:, :1]
    r, grad, ab = loss_and_grad(orc, g, pts, gp, gi)
    assert np.all(np.abs(grad[:, 6:10]) <= 1e-12 * (1 + np.abs(grad[:, 0:3]).max()))
    # the same Gaussians made anisotropic do get a rotation gradient
    g.scale[:, 1] *= np.float32(1.5)
    _, grad2, _ = loss_and_grad(orc, g, pts, gp, gi)
    assert np.abs(grad2[:, 6:10]).max() > 1e-3


def test_quaternion_gradient_orthogonal_to_q(orc):
    """L depends on q only through q/|q|: dL/dq is orthogonal to q."""
    g, pts, gp, gi = cluster(24)
    _, grad, ab = loss_and_grad(orc, g, pts, gp, gi)
    dots = np.sum(grad[:, 6:10] * g.rot.astype(np.float64), axis=1)
    assert np.all(np.abs(dots) <= 1e-10 * (1 + ab[:, 6:10].sum(axis=1)))


def test_undefined_and_masked_points_carry_no_gradient(orc):
    g, pts, gp, gi = cluster(25)
    r = orc.forward(g, pts)
    und = ~r.defined.astype(bool)
    assert und.sum() > 100
    grad_all, _ = orc.backward(g, pts, r.phi, r.inf, gp, gi)
    gp2, gi2 = gp.copy(), gi.copy()
    gp2[und] = 123.0
    gi2[und] = -77.0
    grad2, _ = orc.backward(g, pts, r.phi, r.inf, gp2, gi2)
    np.testing.assert_array_equal(grad_all, grad2)
    mask = np.zeros(len(pts), dtype=np.uint8)
    mask[::2] = 1
    gm, _ = orc.backward(g, pts, r.phi, r.inf, gp, gi, zero_mask=mask)
    gp3, gi3 = gp.copy(), gi.copy()
    gp3[::2] = 0
    gi3[::2] = 0
    g3, _ = orc.backward(g, pts, r.phi, r.inf, gp3, gi3)
    np.testing.assert_allclose(gm, g3, rtol=0, atol=1e-13)


def test_selection_and_prune_match_full(orc):
    g, pts, gp, gi = cluster(26)
    r = orc.forward(g, pts)
    full, fab = orc.backward(g, pts, r.phi, r.inf, gp, gi)
    sel = np.array([3, 0, 17, 5])
    part, pab = orc.backward(g, pts, r.phi, r.inf, gp, gi, select=sel)
    np.testing.assert_array_equal(part, full[sel])
    np.testing.assert_array_equal(pab, fab[sel])
    nop, _ = orc.backward(g, pts, r.phi, r.inf, gp, gi, prune=False)
    np.testing.assert_array_equal(nop, full)
    # support: points out of every selected Gaussian's reach do not matter
    sup = orc.support(g, pts, sel)
    part2, _ = orc.backward(g, pts[sup], r.phi[sup], r.inf[sup], gp[sup], gi[sup], select=sel)
    np.testing.assert_allclose(part2, part, rtol=1e-12, atol=1e-14)


def loss(orc, g, pts, gp, gi):
    r = orc.forward(g, pts)
    return float(np.sum(gp * r.phi + gi * r.inf)), r


def perturbed(g, field, i, k, delta):
    arrs = {f: getattr(g, f).astype(np.float64).copy() for f in ("mean", "scale", "rot", "value", "weight")}
    a = arrs[field]
    if a.ndim == 1:
        a[i] += delta
    else:
        a[i, k] += delta
    return synth.Gaussians(arrs["mean"], arrs["scale"], arrs["rot"], arrs["value"], arrs["weight"])


@pytest.mark.parametrize("seed", [31, 32])
def test_central_finite_differences(orc, seed):
    """Every one of the 12 gradient entries of several Gaussians against
    central differences of the float64 forward, skipping draws where the
    step flips an inclusion or a definedness."""
    g, pts, gp, gi = cluster(seed, n=12, npts=1500)
    g64 = synth.Gaussians(*(getattr(g, f).astype(np.float64) for f in ("mean", "scale", "rot", "value", "weight")))
    L0, r0 = loss(orc, g64, pts, gp, gi)
    grad, ab = orc.backward(g64, pts, r0.phi, r0.inf, gp, gi)
    layout = [("mean", k) for k in range(3)] + [("scale", k) for k in range(3)] + \
             [("rot", k) for k in range(4)] + [("value", None), ("weight", None)]
    checked = 0
    for i in range(12):
        for col, (field, k) in enumerate(layout):
            base = getattr(g64, field)[i] if k is None else getattr(g64, field)[i, k]
            h = 1e-6 * max(abs(base), 0.05 if field in ("mean", "scale") else 1.0)
            Lp, rp = loss(orc, perturbed(g64, field, i, k, h), pts, gp, gi)
            Lm, rm = loss(orc, perturbed(g64, field, i, k, -h), pts, gp, gi)
            if not (np.array_equal(rp.ncontrib, r0.ncontrib) and np.array_equal(rm.ncontrib, r0.ncontrib) and
                    np.array_equal(rp.defined, r0.defined) and np.array_equal(rm.defined, r0.defined)):
                continue
            fd = (Lp - Lm) / (2 * h)
            tol = 1e-6 * (abs(grad[i, col]) + ab[i, col]) + 1e-13 * max(1.0, abs(L0)) / h
            assert abs(fd - grad[i, col]) <= tol, (i, field, k, fd, grad[i, col], ab[i, col])
            checked += 1
    assert checked >= 12 * 12 * 0.8
