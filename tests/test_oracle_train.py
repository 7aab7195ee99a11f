"""Pins of the oracle's training epilogue: the activations of Sec. 4.2 and
the L1 / false-negative (Eq. 4) / false-positive (Eq. 5) losses with their
cotangents. Checked against a batch worked by hand, closed forms of the
activations, limits and invariants, and central finite differences."""
import math
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def load_golden():
    params, terms, counts, rows = {}, None, None, []
    for line in open(os.path.join(HERE, "golden", "loss_small.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        f = line.split()
        if f[0] == "params":
            params = {k: float(v) for k, v in (x.split("=") for x in f[1:])}
        elif f[0] == "terms":
            terms = [float(x) for x in f[1:]]
        elif f[0] == "counts":
            counts = [int(x) for x in f[1:]]
        else:
            rows.append([float(x) for x in f])
    return params, terms, counts, np.array(rows)


def test_loss_hand_worked_batch():
    p, terms, counts, rows = load_golden()
    r = oracle.loss(rows[:, 0], rows[:, 1], rows[:, 2], rows[:, 3].astype(np.uint8), tau=p["tau"], eps=p["eps"],
                    lambda_fn=p["lambda_fn"], lambda_fp=p["lambda_fp"])
    assert [r.l1, r.fn, r.fp, r.total] == terms
    assert [r.n_defined, r.n_fn, r.n_fp] == counts
    np.testing.assert_array_equal(r.grad_value, rows[:, 4].astype(np.float32))
    np.testing.assert_array_equal(r.grad_influence, rows[:, 5].astype(np.float32))


def test_loss_without_flags_means_every_sample_is_in_the_volume():
    p, _, _, rows = load_golden()
    kw = dict(tau=p["tau"], eps=p["eps"], lambda_fn=p["lambda_fn"], lambda_fp=p["lambda_fp"])
    a = oracle.loss(rows[:4, 0], rows[:4, 1], rows[:4, 2], None, **kw)
    b = oracle.loss(rows[:4, 0], rows[:4, 1], rows[:4, 2], np.ones(4, np.uint8), **kw)
    assert (a.l1, a.fn, a.fp, a.total) == (b.l1, b.fn, b.fp, b.total) == (0.28125, 0.109375, 0.0, 0.390625)
    np.testing.assert_array_equal(a.grad_value, b.grad_value)
    np.testing.assert_array_equal(a.grad_influence, b.grad_influence)


def batch(seed, n, tau=0.01, frac_undef=0.2, frac_out=0.2):
    g = np.random.default_rng(seed)
    phi = g.random(n).astype(np.float32)
    inf = (tau * (1.0 + 3.0 * g.random(n))).astype(np.float32)  # I in (tau, 4 tau)
    undef = g.random(n) < frac_undef
    phi[undef] = 0.0
    inf[undef] = 0.0
    y = g.random(n).astype(np.float32)
    dflag = (g.random(n) >= frac_out).astype(np.uint8)
    return phi, inf, y, dflag


def test_loss_empty_sets_and_zero_lambdas():
    n = 50
    z = np.zeros(n, np.float32)
    y = np.linspace(0.0, 1.0, n).astype(np.float32)
    # the model is undefined everywhere: L1 is the mean |y|, every sample is a
    # false negative at distance (1 + eps) tau, and no cotangent flows
    r = oracle.loss(z, z, y, None, tau=0.01, eps=0.25, lambda_fn=2.0, lambda_fp=5.0)
    assert r.n_defined == n and r.n_fn == n and r.n_fp == 0
    assert math.isclose(r.l1, float(np.mean(y.astype(np.float64))), rel_tol=1e-15)
    assert math.isclose(r.fn, 2.0 * 1.25 * float(np.float32(0.01)), rel_tol=1e-15)
    assert r.fp == 0.0
    assert not r.grad_value.any() and not r.grad_influence.any()
    # nothing in the volume: only the false-positive term
    phi, inf, y, _ = batch(3, 200)
    r = oracle.loss(phi, inf, y, np.zeros(200, np.uint8), lambda_fn=7.0, lambda_fp=1.0)
    assert r.n_defined == 0 and r.l1 == 0.0 and r.fn == 0.0 and not r.grad_value.any()
    assert math.isclose(r.fp, float(inf[inf > 0].astype(np.float64).mean()), rel_tol=1e-14)
    # lambdas of zero switch their terms and cotangents off
    phi, inf, y, d = batch(4, 300)
    r = oracle.loss(phi, inf, y, d, lambda_fn=0.0, lambda_fp=0.0)
    assert r.fn == 0.0 and r.fp == 0.0 and not r.grad_influence.any()
    # an empty batch
    e = np.zeros(0, np.float32)
    r = oracle.loss(e, e, e, None)
    assert (r.l1, r.fn, r.fp, r.total) == (0.0, 0.0, 0.0, 0.0)


def test_loss_permutation():
    phi, inf, y, d = batch(5, 400)
    a = oracle.loss(phi, inf, y, d)
    pm = np.random.default_rng(9).permutation(400)
    b = oracle.loss(phi[pm], inf[pm], y[pm], d[pm])
    assert (a.n_defined, a.n_fn, a.n_fp) == (b.n_defined, b.n_fn, b.n_fp)
    for x, z in ((a.l1, b.l1), (a.fn, b.fn), (a.fp, b.fp)):
        assert math.isclose(x, z, rel_tol=1e-13)
    np.testing.assert_array_equal(a.grad_value[pm], b.grad_value)
    np.testing.assert_array_equal(a.grad_influence[pm], b.grad_influence)


def test_loss_cotangents_are_the_derivative():
    """Central differences of the float64 loss in one output at a time (the
    set memberships stay fixed for a small step away from the thresholds)."""
    tau, eps, lfn, lfp = 0.01, 0.5, 3.0, 2.0
    phi, inf, y, d = batch(6, 64)
    r = oracle.loss(phi, inf, y, d, tau=tau, eps=eps, lambda_fn=lfn, lambda_fp=lfp)
    thr = (1.0 + eps) * float(np.float32(tau))
    h = 2.0 ** -20

    def total(phi_, inf_):
        # the oracle takes float32; evaluate at float64 steps with the same
        # memberships by computing the smooth pieces from its set sizes
        q = oracle.loss(phi_, inf_, y, d, tau=tau, eps=eps, lambda_fn=lfn, lambda_fp=lfp)
        assert (q.n_defined, q.n_fn, q.n_fp) == (r.n_defined, r.n_fn, r.n_fp)
        return q.total

    checked = 0
    for i in range(64):
        if inf[i] == 0.0:
            assert r.grad_value[i] == 0.0 and r.grad_influence[i] == 0.0
            continue
        if abs(phi[i] - y[i]) > 4 * h and d[i]:
            p1, p0 = phi.copy(), phi.copy()
            p1[i] += h
            p0[i] -= h
            num = (total(p1, inf) - total(p0, inf)) / (float(p1[i]) - float(p0[i]))
            assert math.isclose(num, float(r.grad_value[i]), rel_tol=1e-6), (i, num, r.grad_value[i])
            checked += 1
        if abs(float(inf[i]) - thr) > 4 * h and abs(float(inf[i]) - tau) > 4 * h:
            i1, i0 = inf.copy(), inf.copy()
            i1[i] += h
            i0[i] -= h
            num = (total(phi, i1) - total(phi, i0)) / (float(i1[i]) - float(i0[i]))
            assert abs(num - float(r.grad_influence[i])) <= 1e-6 * max(1.0, abs(num)), (i, num, r.grad_influence[i])
            checked += 1
    assert checked > 60


def raw(seed, n, mu=math.log(0.008), sd=0.4):
    g = np.random.default_rng(seed)
    return oracle.RawGaussians(g.normal(mu, sd, (n, 3)), g.normal(0, 2, n), g.normal(0, 2, n))


def test_sigmoid_closed_forms():
    r = oracle.RawGaussians(np.zeros((3, 3)), [0.0, math.log(3.0), -math.log(3.0)], [0.0, -math.log(3.0), 50.0])
    _, v, w = oracle.activate(r, 0.0)
    np.testing.assert_allclose(v, [0.5, 0.75, 0.25], rtol=1e-15)
    assert w[0] == 0.5 and math.isclose(w[1], 0.25, rel_tol=1e-15) and 1.0 - w[2] < 1e-20
    _, dv, dw = oracle.activate_backward(r, 0.0, np.zeros((3, 3)), np.ones(3), np.ones(3))
    np.testing.assert_allclose(dv, [0.25, 0.1875, 0.1875], rtol=1e-15)
    assert dw[0] == 0.25
    # far in the tail the derivative is e^-x (1 + O(e^-x)), not a rounded 0
    r = oracle.RawGaussians(np.zeros((2, 3)), [40.0, -60.0], [80.0, 700.0])
    _, dv, dw = oracle.activate_backward(r, 0.0, np.zeros((2, 3)), np.ones(2), np.ones(2))
    np.testing.assert_allclose(dv, [math.exp(-40.0), math.exp(-60.0)], rtol=1e-15)
    np.testing.assert_allclose(dw, [math.exp(-80.0), math.exp(-700.0)], rtol=1e-15)


def test_scale_without_cap_is_exp():
    r = raw(1, 100)
    s, _, _ = oracle.activate(r, 0.0)
    np.testing.assert_allclose(s, np.exp(r.log_scale), rtol=5e-16)  # libm and numpy exp differ by an ulp
    s2, _, _ = oracle.activate(r, -1.0)
    np.testing.assert_array_equal(s2, s)


def test_soft_cap_closed_forms():
    c = 0.02
    d = np.array([1.0, 2.0, 2.0]) / 3.0  # unit direction
    # |e| = c atanh(1/2): the capped norm is exactly c / 2, along e
    e = d * c * math.atanh(0.5)
    s, _, _ = oracle.activate(oracle.RawGaussians(np.log(e)[None], [0.0], [0.0]), c)
    assert math.isclose(np.linalg.norm(s[0]), c / 2, rel_tol=1e-14)
    np.testing.assert_allclose(s[0] / np.linalg.norm(s[0]), d, rtol=1e-14)
    # far above the cap the norm tends to c, and never exceeds it
    for k in (2.0, 10.0, 1e3):
        s, _, _ = oracle.activate(oracle.RawGaussians(np.log(d * c * k)[None], [0.0], [0.0]), c)
        nrm = np.linalg.norm(s[0])
        assert nrm <= c and math.isclose(nrm, c * math.tanh(k), rel_tol=1e-13)  # tanh(1000) rounds to 1
    # far below the cap it is the identity to first order: s = e (1 - |e|^2 / (3 c^2)) + O(|e|^4)
    for k in (1e-1, 1e-2, 1e-3, 1e-5):
        e = d * c * k
        s, _, _ = oracle.activate(oracle.RawGaussians(np.log(e)[None], [0.0], [0.0]), c)
        assert np.all(np.abs(s[0] / e - (1.0 - k * k / 3.0)) <= 0.2 * k ** 4 + 1e-15)


def test_soft_cap_monotone_along_a_ray():
    c = 0.04
    d = np.array([0.3, 0.5, 0.2])
    d /= np.linalg.norm(d)
    ks = np.geomspace(1e-4, 10.0, 200)
    logs = np.log(d[None, :] * c * ks[:, None])
    s, _, _ = oracle.activate(oracle.RawGaussians(logs, np.zeros(200), np.zeros(200)), c)
    nrm = np.linalg.norm(s, axis=1)
    assert np.all(np.diff(nrm) > 0) and np.all(nrm < c)


@pytest.mark.parametrize("cap", [0.0, 0.02, 0.04])
def test_activation_backward_finite_differences(cap):
    n = 40
    r = raw(2, n, mu=math.log(0.01), sd=1.5)  # norms from far below to far above the cap
    g = np.random.default_rng(8)
    ds, dv, dw = g.standard_normal((n, 3)), g.standard_normal(n), g.standard_normal(n)
    a, b, c_ = oracle.activate_backward(r, cap, ds, dv, dw)

    def Ls(rr):  # per Gaussian; the parts are differenced apart so that
        s, _, _ = oracle.activate(rr, cap)  # rounding of the large sigmoid terms
        return (s * ds).sum(axis=1)         # does not swamp the small scale terms

    def L(rr):
        _, v, w = oracle.activate(rr, cap)
        return v * dv + w * dw

    h = 1e-6
    for k in range(3):
        lp = r.log_scale.copy()
        lm = r.log_scale.copy()
        lp[:, k] += h
        lm[:, k] -= h
        num = (Ls(oracle.RawGaussians(lp, r.value_logit, r.weight_logit)) -
               Ls(oracle.RawGaussians(lm, r.value_logit, r.weight_logit))) / (2 * h)
        scale = np.abs(ds).sum(axis=1) * np.exp(r.log_scale).max(axis=1)
        assert np.all(np.abs(num - a[:, k]) <= 1e-8 * scale + 1e-12 * np.abs(a[:, k])), k
    for which in ("v", "w"):
        vp, vm = r.value_logit.copy(), r.value_logit.copy()
        wp, wm = r.weight_logit.copy(), r.weight_logit.copy()
        if which == "v":
            vp += h
            vm -= h
        else:
            wp += h
            wm -= h
        num = (L(oracle.RawGaussians(r.log_scale, vp, wp)) - L(oracle.RawGaussians(r.log_scale, vm, wm))) / (2 * h)
        ref = b if which == "v" else c_
        np.testing.assert_allclose(num, ref, rtol=1e-6, atol=1e-10)


def test_soft_cap_series_meets_closed_form():
    """The factor switches from its series to the closed form at |e| = c/100;
    both sides of the switch agree with the closed form evaluated in long
    double precision (mpmath-free: the difference of two nearby points)."""
    c = 0.02
    d = np.array([0.6, 0.0, 0.8])
    ks = np.array([0.0099999, 0.01, 0.0100001])
    logs = np.log(np.maximum(d[None, :] * c * ks[:, None], 1e-300))
    logs[:, 1] = -700.0  # a zero axis (exp underflows to 0)
    s, _, _ = oracle.activate(oracle.RawGaussians(logs, np.zeros(3), np.zeros(3)), c)
    nrm = np.linalg.norm(s, axis=1)
    ref = c * np.tanh(ks)
    np.testing.assert_allclose(nrm, ref, rtol=1e-13)
    ds = np.tile([1.0, 0.5, -2.0], (3, 1))
    a, _, _ = oracle.activate_backward(oracle.RawGaussians(logs, np.zeros(3), np.zeros(3)), c, ds, np.zeros(3),
                                       np.zeros(3))
    assert np.all(np.abs(np.diff(a[:, 0])) < 1e-4 * np.abs(a[1, 0]))
