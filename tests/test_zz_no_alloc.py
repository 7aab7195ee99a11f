"""The backward entry point that allocates nothing
(gs_sample_backward_noalloc, its workspace a static device array of the
library) against gs_sample_backward with a caller workspace: bit-identical
gradients on consecutive calls, the second with a smaller input, for point
and grid queries."""
import numpy as np
import pytest

import synth
from harness import Run, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def noalloc_grads(r: Run, gv, gi):
    import torch
    import paper_2607_01164_amd as gs
    grads = gs.Grads.empty(r.g.n, "cuda")
    gs.gs_sample_backward_noalloc(r.dg, r.index, r.query, r.plan, r.value, r.influence, r.gv, r.gi, grads)
    torch.cuda.synchronize()
    return np.concatenate([grads.mean.cpu().numpy(), grads.scale.cpu().numpy(), grads.rot.cpu().numpy(),
                           grads.value.cpu().numpy()[:, None], grads.weight.cpu().numpy()[:, None]], axis=1)


def test_noalloc_backward_matches_the_workspace_backward():
    cases = [("points", 70000, 60000, (16, 16, 16), 1), ("points", 3000, 20000, (8, 8, 8), 2),
             ("grid", 2000, 0, (8, 8, 8), 3)]
    for kind, n_gauss, npts, cells, seed in cases:
        g = synth.random_gaussians(300 + seed, n_gauss, log_mu=np.log(0.02 if n_gauss > 10000 else 0.04),
                                   log_sd=0.4)
        log(f"case no-alloc backward: {kind}, {n_gauss} Gaussians, cells {cells}")
        if kind == "points":
            r = Run(g, cells, "points", points=synth.random_points(310 + seed, npts))
        else:
            r = Run(g, cells, "grid", dims=(32, 32, 32))
        r.forward()
        gv, gi = synth.random_normal(320 + seed, r.nq), synth.random_normal(330 + seed, r.nq)
        want = r.backward(gv, gi)
        got = noalloc_grads(r, gv, gi)
        assert np.any(want != 0)
        np.testing.assert_array_equal(got, want)


def test_noalloc_backward_rejects_a_workspace_beyond_its_array():
    import paper_2607_01164_amd as gs
    g = synth.random_gaussians(340, 1000)
    r = Run(g, (8, 8, 8), "points", points=synth.random_points(341, 5_000_000))
    r.forward()
    gv, gi = synth.random_normal(342, r.nq), synth.random_normal(343, r.nq)
    r.backward(gv, gi)
    with pytest.raises(gs.GsError) as e:
        noalloc_grads(r, gv, gi)
    assert e.value.status == gs.GS_ERR_WORKSPACE
