"""Pins of the oracle's forward pass (Eq. 2, Eq. 3, cutoff of Sec. 4.1.1,
definedness of Sec. 4.1.3, domain culling of Sec. 5) against closed forms,
invariants and an independent scipy-based twin. CPU only."""
import math
import os

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TAU = 0.01
T = 2.0 * math.log(100.0)


def one(mean, scale, rot, value, weight, dtype=np.float32):
    return synth.Gaussians(np.asarray([mean], dtype), np.asarray([scale], dtype), np.asarray([rot], dtype),
                           np.asarray([value], dtype), np.asarray([weight], dtype))


def concat(*gs):
    return synth.Gaussians(*(np.concatenate([getattr(g, f) for g in gs]) for f in
                             ("mean", "scale", "rot", "value", "weight")))


def unit_dirs(seed, n):
    d = np.random.default_rng(seed).standard_normal((n, 3))
    return d / np.linalg.norm(d, axis=1, keepdims=True)


def load_isotropic():
    rows = []
    with open(os.path.join(GOLDEN, "isotropic_single.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(x) for x in line.split()])
    return np.asarray(rows)


def test_isotropic_single_gaussian_radii(orc):
    """Closed form of a single isotropic Gaussian at known Mahalanobis radii,
    for several rotations: I = w exp(-r^2/2), Phi = v, undefined beyond
    sqrt(2 ln(w/tau)), excluded beyond the cutoff radius."""
    rows = load_isotropic()
    sigma, mu = 0.0625, np.array([0.5, 0.5, 0.5])
    v32 = float(np.float32(0.7))
    rots = [(1, 0, 0, 0), (0.3, -0.5, 0.2, 0.9), (0, 0, 0, 1), (-0.7, 0.1, 0.1, 0.7)]
    for q in rots:
        g = one(mu, (sigma,) * 3, q, 0.7, 0.5)
        dirs = unit_dirs(1, 16)
        for r, eI, ePhi, dfd, hit in rows:
            pts = mu[None, :] + r * sigma * dirs
            res = orc.forward(g, pts, tau=TAU)
            assert np.all(res.defined == int(dfd))
            assert np.all(res.ncontrib == int(hit))
            np.testing.assert_allclose(res.inf, eI, rtol=1e-12, atol=0)
            np.testing.assert_allclose(res.phi, v32 if dfd else 0.0, rtol=1e-12, atol=0)


def test_two_gaussians_closed_form(orc):
    """Eq. 2 for two isotropic Gaussians along x, written as a direct sum."""
    s1, s2 = 0.05, 0.08
    g = concat(one((0.4, 0.5, 0.5), (s1,) * 3, (1, 0, 0, 0), 0.2, 0.3),
               one((0.6, 0.5, 0.5), (s2,) * 3, (0.6, 0.0, 0.8, 0.0), 0.8, 0.9))
    xs = np.linspace(0.2, 0.85, 131)
    pts = np.stack([xs, np.full_like(xs, 0.5), np.full_like(xs, 0.52)], axis=1)
    res = orc.forward(g, pts, tau=TAU)
    m = g.mean.astype(np.float64)
    s = np.array([np.float64(np.float32(s1)), np.float64(np.float32(s2))])
    w = g.weight.astype(np.float64)
    v = g.value.astype(np.float64)
    for p, ph, inf, dfd in zip(pts, res.phi, res.inf, res.defined):
        r2 = np.sum((p[None, :] - m) ** 2, axis=1) / s ** 2
        Gs = np.where(r2 <= T, np.exp(-0.5 * r2), 0.0)
        I = np.sum(w * Gs)
        if I > np.float32(TAU):
            assert dfd == 1
            assert inf == pytest.approx(I, rel=1e-12)
            assert ph == pytest.approx(np.sum(w * v * Gs) / I, rel=1e-12)
        else:
            assert dfd == 0 and inf == 0.0 and ph == 0.0


def test_spherical_rotation_invariance(orc):
    """A spherical Gaussian's field does not depend on its quaternion."""
    pts = synth.random_points(5, 4000, 0.3, 0.7)
    outs = []
    for q in [(1, 0, 0, 0), (0.1, 0.2, 0.3, 0.4), (-3, 1, 0.5, 2), (0, 1, 0, 0)]:
        g = concat(one((0.5, 0.5, 0.5), (0.05,) * 3, q, 0.4, 0.8), one((0.55, 0.45, 0.5), (0.04, 0.04, 0.04), q, 0.9, 0.3))
        outs.append(orc.forward(g, pts))
    for r in outs[1:]:
        np.testing.assert_array_equal(r.defined, outs[0].defined)
        np.testing.assert_allclose(r.inf, outs[0].inf, rtol=1e-13, atol=0)
        np.testing.assert_allclose(r.phi, outs[0].phi, rtol=1e-13, atol=0)


def test_rotation_convention_pin(orc):
    """s = (a, b, c) with b << a and a 90 degree turn about z: the long axis
    moves from x to y, i.e. G(mu + r a y) = exp(-r^2/2) and the same offset
    along x lands far outside. Pins R(q) (Hamilton, w first) and Eq. 3's
    reading Sigma = R S^2 R^T."""
    a, b, c = 0.1, 0.01, 0.02
    h = math.sqrt(0.5)
    mu = np.array([0.5, 0.5, 0.5])
    g = one(mu, (a, b, c), (h, 0, 0, h), 0.3, 1.0)
    a32 = float(np.float32(a))
    for r in (0.0, 0.5, 1.0, 2.0):
        res = orc.forward(g, (mu + np.array([0, r * a32, 0]))[None, :])
        assert res.inf[0] == pytest.approx(math.exp(-r * r / 2), rel=1e-6)
        if r > 0:
            res_x = orc.forward(g, (mu + np.array([r * a32, 0, 0]))[None, :])
            assert res_x.ncontrib[0] == 0 and res_x.inf[0] == 0.0
    # local z stays world z
    res_z = orc.forward(g, (mu + np.array([0, 0, float(np.float32(c))]))[None, :])
    assert res_z.inf[0] == pytest.approx(math.exp(-0.5), rel=1e-6)


def test_phi_within_value_range_and_constant_values(orc):
    g = synth.random_gaussians(11, 200, log_mu=np.log(0.06))
    g.value[:] = np.float32(0.2) + np.float32(0.6) * g.value
    pts = synth.random_points(11, 5000)
    r = orc.forward(g, pts)
    d = r.defined.astype(bool)
    assert d.sum() > 1000
    assert np.all(r.phi[d] >= g.value.min() - 1e-12) and np.all(r.phi[d] <= g.value.max() + 1e-12)
    g.value[:] = np.float32(0.37)
    r2 = orc.forward(g, pts)
    np.testing.assert_allclose(r2.phi[d], np.float64(np.float32(0.37)), rtol=1e-13)
    np.testing.assert_array_equal(r2.inf, r.inf)


def test_permutation_invariance(orc):
    g = synth.random_gaussians(12, 150, log_mu=np.log(0.06))
    pts = synth.random_points(12, 3000)
    r = orc.forward(g, pts)
    perm = np.random.default_rng(3).permutation(150)
    r2 = orc.forward(g.subset(perm), pts)
    np.testing.assert_array_equal(r.defined, r2.defined)
    np.testing.assert_allclose(r2.inf, r.inf, rtol=1e-13)
    np.testing.assert_allclose(r2.phi, r.phi, rtol=1e-13)


def test_weight_scaling_invariance(orc):
    """Scaling every weight by c scales I by c and leaves Phi unchanged where
    the point stays defined (the cutoff ignores w)."""
    g = synth.random_gaussians(13, 150, log_mu=np.log(0.06))
    pts = synth.random_points(13, 3000)
    r = orc.forward(g, pts)
    g2 = synth.Gaussians(g.mean, g.scale, g.rot, g.value, (g.weight * np.float32(0.5)).astype(np.float32))
    r2 = orc.forward(g2, pts)
    np.testing.assert_array_equal(r.ncontrib, r2.ncontrib)
    both = r.defined.astype(bool) & r2.defined.astype(bool)
    assert both.sum() > 500
    np.testing.assert_allclose(r2.phi[both], r.phi[both], rtol=1e-12)
    np.testing.assert_allclose(r2.inf[both], 0.5 * r.inf[both], rtol=1e-12)


def test_split_into_copies_leaves_eq2_unchanged(orc):
    """Replacing a Gaussian by n copies with weight w/n leaves Eq. 2 exactly
    as it was (the MCMC relocation rule of Sec. 4.2.1)."""
    g = synth.random_gaussians(14, 60, log_mu=np.log(0.08))
    g.weight[:] = np.float32(0.75)
    pts = synth.random_points(14, 3000)
    r = orc.forward(g, pts)
    idx = np.concatenate([np.arange(60), [7, 7, 23, 23, 23]])
    gs = g.subset(idx)
    gs.weight = gs.weight.copy()
    gs.weight[[7, 60, 61]] = np.float32(0.25)        # 3 copies of #7, w/3
    gs.weight[[23, 62, 63, 64]] = np.float32(0.1875)  # 4 copies of #23, w/4
    r2 = orc.forward(gs, pts)
    np.testing.assert_array_equal(r.defined, r2.defined)
    np.testing.assert_allclose(r2.inf, r.inf, rtol=1e-12)
    np.testing.assert_allclose(r2.phi, r.phi, rtol=1e-12)


def test_out_of_domain_and_empty_space(orc):
    g = concat(one((0.0, 0.5, 0.5), (0.05,) * 3, (1, 0, 0, 0), 0.5, 0.9),
               one((1.0, 1.0, 1.0), (0.05,) * 3, (1, 0, 0, 0), 0.5, 0.9))
    pts = np.array([[-0.01, 0.5, 0.5],     # covered but outside the box
                    [0.0, 0.5, 0.5],       # on the closed boundary: inside
                    [0.01, 0.5, 0.5],
                    [1.0, 1.0, 1.0],
                    [1.0 + 1e-6, 1.0, 1.0],
                    [0.5, 0.5, 0.5],       # empty space
                    [0.5, 0.0, 0.0]])
    r = orc.forward(g, pts)
    assert list(r.defined) == [0, 1, 1, 1, 0, 0, 0]
    assert r.phi[0] == 0.0 and r.inf[0] == 0.0 and r.phi[4] == 0.0 and r.inf[4] == 0.0
    assert r.ncontrib[5] == 0 and r.inf[5] == 0.0
    assert r.inf[1] == pytest.approx(float(np.float32(0.9)), rel=1e-12)
    # a box other than the unit cube
    r2 = orc.forward(g, pts, lo=(-0.1, 0, 0), hi=(1.1, 1.1, 1.1))
    assert r2.defined[0] == 1 and r2.defined[4] == 1


def test_invalid_gaussians_contribute_nothing(orc):
    good = one((0.5, 0.5, 0.5), (0.05,) * 3, (1, 0, 0, 0), 0.5, 0.9)
    bad = [one((0.5, 0.5, 0.5), (0.05,) * 3, (0, 0, 0, 0), 0.5, 0.9),
           one((0.5, 0.5, 0.5), (0.05, 0.0, 0.05), (1, 0, 0, 0), 0.5, 0.9),
           one((0.5, np.nan, 0.5), (0.05,) * 3, (1, 0, 0, 0), 0.5, 0.9),
           one((0.5, 0.5, 0.5), (0.05,) * 3, (1, 0, 0, 0), np.inf, 0.9),
           one((0.5, 0.5, 0.5), (0.05, -0.05, 0.05), (1, 0, 0, 0), 0.5, 0.9)]
    pts = synth.random_points(3, 500, 0.4, 0.6)
    r0 = orc.forward(good, pts)
    r1 = orc.forward(concat(good, *bad), pts)
    np.testing.assert_array_equal(r0.inf, r1.inf)
    np.testing.assert_array_equal(r0.phi, r1.phi)


def test_prune_is_exact(orc):
    g = synth.random_gaussians(15, 300, log_mu=np.log(0.04), log_sd=0.7)
    pts = synth.random_points(15, 4000)
    a = orc.forward(g, pts, prune=True)
    b = orc.forward(g, pts, prune=False)
    for f in ("phi", "inf", "defined", "ncontrib", "namb", "b_phi", "b_inf"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))


def scipy_twin(g, pts, lo=(0, 0, 0), hi=(1, 1, 1), tau=TAU):
    """Independent float64 Eq. 2 through scipy's quaternion rotations and the
    inverse covariance (conic form); quaternions are normalised by scipy."""
    from scipy.spatial.transform import Rotation
    q = g.rot.astype(np.float64)
    R = Rotation.from_quat(np.stack([q[:, 1], q[:, 2], q[:, 3], q[:, 0]], axis=1)).as_matrix()
    S2 = g.scale.astype(np.float64) ** 2
    cov = np.einsum("nij,nj,nkj->nik", R, S2, R)
    icov = np.linalg.inv(cov)
    mu = g.mean.astype(np.float64)
    d = pts[:, None, :].astype(np.float64) - mu[None, :, :]
    Q = np.einsum("pni,nij,pnj->pn", d, icov, d)
    Tc = 2.0 * np.log(1.0 / np.float64(np.float32(tau)))
    G = np.where(Q <= Tc, np.exp(-0.5 * Q), 0.0)
    w = g.weight.astype(np.float64)
    v = g.value.astype(np.float64)
    I = G @ w
    V = G @ (w * v)
    inside = np.all((pts >= np.asarray(lo)) & (pts <= np.asarray(hi)), axis=1)
    dfd = inside & (I > np.float64(np.float32(tau)))
    return np.where(dfd, V / np.where(dfd, I, 1.0), 0.0), np.where(dfd, I, 0.0), dfd, Q


def test_scipy_twin(orc):
    g = synth.random_gaussians(16, 40, log_mu=np.log(0.08), log_sd=0.5)
    pts = synth.random_points(16, 3000)
    r = orc.forward(g, pts)
    phi, inf, dfd, Q = scipy_twin(g, pts.astype(np.float64))
    amb = orc.ambiguous_points(r)
    ok = ~amb
    assert ok.sum() > 2900
    np.testing.assert_array_equal(r.defined[ok].astype(bool), dfd[ok])
    np.testing.assert_allclose(r.inf[ok], inf[ok], rtol=1e-9, atol=0)
    np.testing.assert_allclose(r.phi[ok], phi[ok], rtol=1e-9, atol=0)
    np.testing.assert_array_equal(r.ncontrib[ok], (Q[ok] <= T).sum(axis=1))


def test_ambiguity_band_flags(orc):
    """Pairs placed exactly at the cutoff radius are ambiguous; pairs at
    r = 0.99 r_c are not."""
    rc = math.sqrt(T)
    mu = np.array([0.5, 0.5, 0.5])
    g = one(mu, (0.05,) * 3, (1, 0, 0, 0), 0.5, 0.9)
    s32 = float(np.float32(0.05))
    pts = np.array([mu + [rc * s32, 0, 0], mu + [0, 0.99 * rc * s32, 0]])
    r = orc.forward(g, pts)
    assert list(r.namb) == [1, 0]
    assert r.amb_a[0, 0] == pytest.approx(0.9 * 0.01 * 1.0, rel=1e-6)


def test_voxel_centers_exact(orc):
    c = orc.voxel_centers((8, 4, 2))
    assert c.shape == (64, 3)
    ids = np.arange(64)
    exp = np.stack([(ids % 8 + 0.5) / 8, ((ids // 8) % 4 + 0.5) / 4, (ids // 32 + 0.5) / 2], axis=1)
    np.testing.assert_array_equal(c, exp.astype(np.float32))
    sub = orc.voxel_centers((8, 4, 2), ids=np.array([5, 63, 0], dtype=np.uint32))
    np.testing.assert_array_equal(sub, exp[[5, 63, 0]].astype(np.float32))
