"""Pins of the oracle's weight pruning and sample-error densification
(Sec. 4.2.1, false negatives first per Sec. 4.2.2): a case worked by hand,
and on random inputs the defining properties checked pair by pair (every
selected sample outranks every eligible one left out, the selection is in
rank order, the kept Gaussians keep their order and parameters)."""
import math
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
TAU_G = 0.0625


def golden():
    gauss, samples, cases = None, [], []
    for line in open(os.path.join(HERE, "golden", "densify_small.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        f = line.split()
        if f[0] == "gauss":
            gauss = np.array([float(x) for x in f[1:]], np.float32)
        elif f[0] == "sample":
            samples.append([float(x) for x in f[1:]])
        elif f[0] == "case":
            cases.append((int(f[1]), int(f[2]), [int(x) for x in f[3:]]))
    return gauss, np.array(samples), cases


def params(n, seed=0):
    g = np.random.default_rng(seed)
    return (g.random((n, 3)).astype(np.float32), g.normal(-4, 0.5, (n, 3)).astype(np.float32),
            g.standard_normal((n, 4)).astype(np.float32), g.standard_normal(n).astype(np.float32),
            g.standard_normal(n).astype(np.float32))


def test_hand_worked_cases():
    w, s, cases = golden()
    m, ls, rot, vl, wl = params(len(w))
    pos = (np.arange(len(s))[:, None] * np.array([0.125, 0.0625, -0.125]) + np.array([0.0, 0.0, 1.0])).astype(
        np.float32)
    for max_new, cap, want in cases:
        r = oracle.densify(m, ls, rot, vl, wl, w, pos, s[:, 4], s[:, 0], s[:, 1], s[:, 2], s[:, 3], tau2=0.005,
                           tau=TAU_G, new_log_scale=-4.0, new_weight_logit=-4.5, max_new=max_new, capacity=cap)
        assert r.n == len(want) and r.source.tolist() == want, (max_new, cap, r.source)
        assert r.kept == 4
        for j, src in enumerate(want):
            if src >= 0:
                np.testing.assert_array_equal(r.mean[j], m[src])
                np.testing.assert_array_equal(r.log_scale[j], ls[src])
                np.testing.assert_array_equal(r.rot[j], rot[src])
                assert r.value_logit[j] == vl[src] and r.weight_logit[j] == wl[src]
            else:
                t = -1 - src
                np.testing.assert_array_equal(r.mean[j], pos[t])
                assert r.log_scale[j].tolist() == [-4.0, -4.0, -4.0]
                assert r.rot[j].tolist() == [1.0, 0.0, 0.0, 0.0] and r.weight_logit[j] == np.float32(-4.5)
                y = min(max(float(s[t, 2]), 2.0 ** -20), 1 - 2.0 ** -20)
                assert r.value_logit[j] == np.float32(math.log(y / (1 - y)))
    # targets 0.75 give logit ln 3; a target of 0 is clamped to 2^-20
    r = oracle.densify(m, ls, rot, vl, wl, w, pos, s[:, 4], s[:, 0], s[:, 1], s[:, 2], s[:, 3], tau2=0.005,
                       tau=TAU_G, max_new=3, capacity=7)
    assert r.value_logit[4] == np.float32(math.log(3.0))
    assert r.value_logit[6] == np.float32(-20 * math.log(2.0) - math.log1p(-2.0 ** -20))
    with pytest.raises(ValueError):
        oracle.densify(m, ls, rot, vl, wl, w, pos, s[:, 4], s[:, 0], s[:, 1], s[:, 2], s[:, 3], tau2=0.005,
                       tau=TAU_G, max_new=1, capacity=3)


def random_case(seed, n_in, nq, tau=0.01):
    g = np.random.default_rng(seed)
    w = g.random(n_in).astype(np.float32) * np.float32(0.02)
    phi = g.random(nq).astype(np.float32)
    inf = (tau * (0.5 + 3 * g.random(nq))).astype(np.float32)
    undef = inf <= np.float32(tau)
    phi[undef] = 0.0
    inf[g.random(nq) < 0.1] = 0.0
    y = g.random(nq).astype(np.float32)
    y[::7] = np.round(y[::7] * 8) / 8  # many equal errors
    phi[::7] = np.round(phi[::7] * 8) / 8
    d = (g.random(nq) > 0.15).astype(np.uint8)
    valid = (g.random(nq) > 0.05).astype(np.uint8)
    pos = g.random((nq, 3)).astype(np.float32)
    return w, phi, inf, y, d, valid, pos


@pytest.mark.parametrize("seed,max_new,cap_extra", [(1, 50, 1000), (2, 500, 30), (3, 10000, 10 ** 6), (4, 0, 5)])
def test_selection_properties(seed, max_new, cap_extra):
    n_in, nq, tau = 300, 700, 0.01
    w, phi, inf, y, d, valid, pos = random_case(seed, n_in, nq, tau)
    m, ls, rot, vl, wl = params(n_in, seed)
    kept = int(np.count_nonzero(w >= np.float32(0.005)))
    cap = kept + cap_extra
    r = oracle.densify(m, ls, rot, vl, wl, w, pos, valid, phi, inf, y, d, tau2=0.005, tau=tau, max_new=max_new,
                       capacity=cap)
    # pruning keeps exactly the heavy-enough Gaussians, in order
    assert r.kept == kept
    np.testing.assert_array_equal(r.source[:kept], np.nonzero(w >= np.float32(0.005))[0])
    eligible = np.nonzero((d != 0) & (valid != 0))[0]
    k = r.n - kept
    assert k == min(max_new, cap - kept, len(eligible))
    sel = -1 - r.source[kept:]
    assert len(set(sel.tolist())) == k and set(sel.tolist()) <= set(eligible.tolist())
    fn = ~(inf > np.float32(tau))
    err = np.abs(phi - y)  # float32, as the ranking takes it

    def outranks(a, b):
        if fn[a] != fn[b]:
            return bool(fn[a])
        if err[a] != err[b]:
            return bool(err[a] > err[b])
        return a < b

    rest = np.setdiff1d(eligible, sel)
    for a in sel:
        for b in rest:
            assert outranks(a, b), (a, b)
    for a, b in zip(sel[:-1], sel[1:]):
        assert outranks(a, b)


def test_without_flags_every_valid_sample_is_eligible():
    w, phi, inf, y, d, valid, pos = random_case(5, 50, 200)
    m, ls, rot, vl, wl = params(50, 5)
    a = oracle.densify(m, ls, rot, vl, wl, w, pos, valid, phi, inf, y, None, max_new=1000, capacity=10 ** 4)
    b = oracle.densify(m, ls, rot, vl, wl, w, pos, valid, phi, inf, y, np.ones(200, np.uint8), max_new=1000,
                       capacity=10 ** 4)
    np.testing.assert_array_equal(a.source, b.source)
    assert a.n - a.kept == int(valid.sum())


def test_nothing_to_prune_or_add():
    m, ls, rot, vl, wl = params(10, 6)
    w = np.full(10, 0.5, np.float32)
    e = np.zeros(0, np.float32)
    r = oracle.densify(m, ls, rot, vl, wl, w, np.zeros((0, 3), np.float32), np.zeros(0, np.uint8), e, e, e, None,
                       max_new=5, capacity=10)
    assert r.n == 10 and r.source.tolist() == list(range(10))
    np.testing.assert_array_equal(r.mean, m)
    r = oracle.densify(m, ls, rot, vl, wl, np.zeros(10, np.float32), np.zeros((0, 3), np.float32),
                       np.zeros(0, np.uint8), e, e, e, None, max_new=5, capacity=10)
    assert r.n == 0
