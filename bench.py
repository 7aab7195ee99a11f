"""Benchmark of the Gaussian-field sampling hot path on one MI355X.

Headline workload: the unstructured training step of the largest
configuration with a backward. 8,388,608 points drawn from a seeded
64-component anisotropic mixture on [0,1]^3 with a spherical cavity of
radius 0.2 left empty, 524,288 Gaussians with means from the same density
and log-scales N(ln 0.005, 0.8) per axis, index 64^3 cells. One step runs
the cloud as four batches of 2^21 points, each a training iteration: build
the cell index, sample (query ordering + forward) and backpropagate N(0,1)
cotangents to every Gaussian parameter. All inputs are resident in HBM
before the timed region.

Prints one JSON line: fwd+bwd samples/s over the timed steps, the per-kernel
timing of the step (HIP events on the library's stream), the roofline of
the dominant kernel, the CPU oracle's rate on a bounded sample of the same
workload, and secondary entries: the 10^8-point full-field forward, the
structured 256^3 batch step, a structured training step (activations,
index, 128^3 jittered samples, losses, backward, activations' backward),
the 32^3 and 512^3 grids, and the point-major against Gaussian-major
forward.
"""
import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_VEC_PEAK_TFLOPS = 157.3   # MI355X vector FP32: 256 CUs x 2.4 GHz x 128 lanes x 2 (packed FMA)
# Algorithmic work of the samplers: a (Gaussian, point) pair that fails the
# cutoff costs the test itself, d = p - mu, u = U d, Q = |u|^2 and the
# compare, counted as 16 operations; a contributing pair costs 30 flops and
# one exponential in the forward (the test, a = w exp(-Q/2), I += a,
# V += a v) and 60 flops and one exponential in the backward (the test, a,
# dL/da, the per-pair moment terms, dv, dw).
FLOPS_FAILING_PAIR = 16.0
FLOPS_CONTRIB = {"sample_points": 31.0, "sample_grid": 31.0, "bwd_gauss": 61.0}
# Bytes one pass of the LSD sort moves per pair: read and write key and value.
SORT_BYTES_PER_PAIR = 16.0
EMIT_BYTES_PER_PAIR = 8.0
COPY_PROBE_BYTES = 256 << 20   # plain copy used to calibrate the HBM byte counters
SRC_DIR = os.path.join(ROOT, "paper_2607_01164_amd", "csrc")
HEADLINE = "c4_points8m"
C2_CELLS = (32, 32, 32)        # the 256^3 batch step's index, the best of a sweep
TRAIN_CELLS = (40, 40, 40)     # the training step's index: twice the batch's query density
TAU = 0.01


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--only", choices=["c4", "c5", "c2", "c3", "c1", "train"], default=None,
                   help="run only this workload's step loop (warmup + steps) and print a short line: for profiling")
    p.add_argument("--cpu-seconds", type=float, default=16.0, help="target length of the CPU oracle sample")
    p.add_argument("--no-cpu", action="store_true")
    p.add_argument("--no-c5", action="store_true", help="skip the 10^8-point full-field forward")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the secondary entries (256^3 batch step, training step, C1, C3, forward A/B)")
    p.add_argument("--breakdown", action="store_true", help="print the per-kernel table to stderr")
    p.add_argument("--copy-probe", action="store_true",
                   help="after the timed region, run a plain 256 MiB copy (counter calibration under rocprofv3)")
    return p.parse_args()


def timed(fn, k, sync):
    sync()
    t0 = time.perf_counter()
    for _ in range(k):
        fn()
    sync()
    return (time.perf_counter() - t0) / k


def kernel_table(gs, fn, k, sync):
    """{kernel: (launches per call, microseconds per call)} over k calls of
    fn with every library kernel bracketed by HIP events (an untimed pass)."""
    gs.profile_select(None)
    gs.profile_reset()
    gs.profile_enable(True)
    for _ in range(k):
        fn()
    sync()
    gs.profile_enable(False)
    return {name: (c / k, ms / k * 1e3) for name, (c, ms) in gs.profile_read().items()}


def kernel_avg_us(gs, name, fn, k, sync):
    """(wall seconds per call, average microseconds per launch of kernel
    `name`) over k timed calls of fn, only that kernel bracketed by HIP
    events on the library's stream."""
    gs.profile_select(name)
    gs.profile_reset()
    gs.profile_enable(True)
    t = timed(fn, k, sync)
    gs.profile_enable(False)
    gs.profile_select(None)
    c, ms = gs.profile_read().get(name, (0, 0.0))
    return t, (ms / c * 1e3 if c else None), c / k


def _dev(torch, np, a, dev="cuda:0"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


class SidePlans:
    """Two plans and a side stream: a step's query ordering (gs_plan_queries)
    runs there while the main stream builds the index and finishes the step
    before; the planned forward waits for it, and a plan is reused once the
    backward that read it has run."""

    def __init__(self, gs, torch, query, grid, dev):
        self.gs, self.torch = gs, torch
        self.plans = [gs.alloc_plan(query, grid, dev) for _ in range(2)]
        self.side = torch.cuda.Stream()
        self.planned = [torch.cuda.Event() for _ in range(2)]
        self.released = [torch.cuda.Event() for _ in range(2)]
        for e in self.released:
            e.record()
        self.k = 0

    def start(self, query, grid):
        k = self.k
        self.side.wait_event(self.released[k])
        with self.torch.cuda.stream(self.side):
            self.gs.gs_plan_queries(query, grid, self.plans[k], stream=self.side)
            self.planned[k].record(self.side)
        return self.plans[k]

    def wait(self):
        self.torch.cuda.current_stream().wait_event(self.planned[self.k])

    def release(self):
        self.released[self.k].record()
        self.k ^= 1


class PointsStep:
    """The unstructured workload's training step: the point cloud in
    `batches` resident batches; each is one iteration of index build,
    forward (query ordering included) and backward with its own N(0,1)
    cotangents. The index is rebuilt every iteration, as training changes
    the Gaussians after each one."""

    def __init__(self, name="c4_points8m"):
        import numpy as np
        import torch

        import paper_2607_01164_amd as gs
        import synth
        self.gs, self.torch, self.np = gs, torch, np
        w = synth.WORKLOADS[name]
        self.w = w
        g = synth.make_gaussians(w)
        self.g_host = g
        pts = synth.make_points(w)
        perm = synth.batch_permutation(w, len(pts))
        self.batches = len(pts) // w.batch
        dev = "cuda:0"
        self.dg = gs.Gaussians(*(_dev(torch, np, a) for a in (g.mean, g.scale, g.rot, g.value, g.weight)))
        self.pts, self.gv, self.gi, self.queries = [], [], [], []
        for b in range(self.batches):
            bp = pts[perm[b * w.batch:(b + 1) * w.batch]]
            if b == 0:
                self.batch0_host = bp
            self.pts.append(_dev(torch, np, bp))
            gv, gi = synth.cotangents(w, w.batch, batch_index=b)
            self.gv.append(_dev(torch, np, gv))
            self.gi.append(_dev(torch, np, gi))
            self.queries.append(gs.Query.pts(self.pts[-1]))
        del pts
        self.n = w.batch
        self.grid = gs.make_grid(w.index_cells)
        probe = gs.build_index(self.dg, self.grid, TAU)
        self.index = gs.Index(self.grid, g.n, int(probe.n_pairs * 1.25) + 4096, dev)
        del probe
        self.sp = SidePlans(gs, torch, self.queries[0], self.grid, dev)
        self.plan = self.sp.plans[0]
        self.val = torch.empty(self.n, device=dev)
        self.inf = torch.empty(self.n, device=dev)
        self.grads = gs.Grads.empty(g.n, dev)
        gs.gs_build_index(self.dg, self.grid, TAU, self.index)
        self.work = gs.alloc_backward_work(self.index, self.queries[0], dev)
        self.b = 0
        torch.cuda.synchronize()

    def build(self):
        self.gs.gs_build_index(self.dg, self.grid, TAU, self.index)

    def forward(self, b=None):
        b = self.b if b is None else b
        self.gs.gs_sample(self.dg, self.index, self.queries[b], self.val, self.inf, self.plan)

    def backward(self, b=None):
        b = self.b if b is None else b
        self.gs.gs_sample_backward(self.dg, self.index, self.queries[b], self.plan, self.val, self.inf, self.gv[b],
                                   self.gi[b], self.grads, self.work)

    def iteration(self):
        """One training iteration: the batch's query ordering on the side
        stream (into the plan the batch before last has released), the index
        build on the main stream meanwhile, then the planned forward and the
        backward."""
        b = self.b
        self.plan = self.sp.start(self.queries[b], self.grid)
        self.build()
        self.sp.wait()
        self.gs.gs_sample_planned(self.dg, self.index, self.queries[b], self.val, self.inf, self.plan)
        self.backward()
        self.sp.release()
        self.b = (self.b + 1) % self.batches

    def step(self):
        for _ in range(self.batches):
            self.iteration()

    def pair_counts(self):
        """Per batch (forward tests, backward tests, contributing pairs),
        counted on the device after each batch's forward."""
        out = []
        for b in range(self.batches):
            self.forward(b)
            t, c = self.gs.sample_pair_counts(self.index, self.queries[b], self.plan, self.work)
            bt = self.gs.backward_pair_count(self.index, self.queries[b], self.plan, self.work)
            out.append((t, bt, c))
        return out


class GridBatchStep:
    """The structured 256^3 batch step: 262,144 Gaussians, a seeded batch of
    2^20 distinct voxel centres; index build + forward + backward."""

    def __init__(self, cells=C2_CELLS):
        import numpy as np
        import torch

        import paper_2607_01164_amd as gs
        import synth
        self.gs, self.torch, self.np = gs, torch, np
        w = synth.WORKLOADS["c2_grid256_batch"]
        self.w = w
        g = synth.make_gaussians(w)
        self.g_host = g
        self.ids_host = synth.voxel_batch(w)
        gv, gi = synth.cotangents(w, len(self.ids_host))
        dev = "cuda:0"
        self.dg = gs.Gaussians(*(_dev(torch, np, a) for a in (g.mean, g.scale, g.rot, g.value, g.weight)))
        self.ids = torch.from_numpy(self.ids_host.view(np.int32)).to(dev)
        self.gv, self.gi = _dev(torch, np, gv), _dev(torch, np, gi)
        self.cells = tuple(cells)
        self.grid = gs.make_grid(cells)
        self.query = gs.Query.voxels(w.dims, self.ids)
        self.n = len(self.ids_host)
        probe = gs.build_index(self.dg, self.grid, TAU)
        self.index = gs.Index(self.grid, g.n, int(probe.n_pairs * 1.25) + 4096, dev)
        del probe
        self.sp = SidePlans(gs, torch, self.query, self.grid, dev)
        self.plan = self.sp.plans[0]
        self.val = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.inf = torch.empty(self.n, dtype=torch.float32, device=dev)
        self.grads = gs.Grads.empty(g.n, dev)
        gs.gs_build_index(self.dg, self.grid, TAU, self.index)
        self.work = gs.alloc_backward_work(self.index, self.query, dev)
        torch.cuda.synchronize()

    def build(self):
        self.gs.gs_build_index(self.dg, self.grid, TAU, self.index)

    def forward(self):
        self.gs.gs_sample(self.dg, self.index, self.query, self.val, self.inf, self.plan)

    def backward(self):
        self.gs.gs_sample_backward(self.dg, self.index, self.query, self.plan, self.val, self.inf, self.gv, self.gi,
                                   self.grads, self.work)

    def step(self):
        """Build + forward + backward, the query ordering on the side stream
        meanwhile (SidePlans)."""
        self.plan = self.sp.start(self.query, self.grid)
        self.build()
        self.sp.wait()
        self.gs.gs_sample_planned(self.dg, self.index, self.query, self.val, self.inf, self.plan)
        self.backward()
        self.sp.release()

    def pair_counts(self):
        self.forward()
        t, c = self.gs.sample_pair_counts(self.index, self.query, self.plan, self.work)
        bt = self.gs.backward_pair_count(self.index, self.query, self.plan, self.work)
        return t, bt, c


class TrainStep:
    """Structured training step (Sec. 4.2, Sec. 4.2.2, Sec. 6.1) over the
    free parameters behind the C2 Gaussians: activations (sigmoid values
    and weights, exp scales with the 0.02 soft norm cap), index build, one
    random position in every voxel of a 128^3 grid (2,097,152 samples),
    forward, L1 + false-negative losses against targets, backward, and the
    activations' backward. The offsets and targets of several iterations
    are drawn beforehand and stay in HBM; each step takes the next set, as
    training draws new positions every iteration."""
    DIMS = (128, 128, 128)
    SETS = 4
    CAP = 0.02
    FN_EPS, FN_LAMBDA, FP_LAMBDA = 0.1, 1.0, 0.0

    def __init__(self, st: "GridBatchStep", cells):
        import numpy as np
        import synth
        gs, torch = st.gs, st.torch
        self.st, self.gs, self.torch = st, gs, torch
        self.n = self.DIMS[0] * self.DIMS[1] * self.DIMS[2]
        dev = "cuda:0"
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        ls, vl, wl = synth.raw_params(st.w)
        self.raw = gs.RawParams(t(ls), t(vl), t(wl))
        ng = st.g_host.n
        self.gauss = gs.Gaussians(st.dg.mean, torch.empty(ng, 3, device=dev), st.dg.rot,
                                  torch.empty(ng, device=dev), torch.empty(ng, device=dev))
        self.offsets = [t(synth.jitter_offsets(st.w.cfg, self.n, it)) for it in range(self.SETS)]
        self.targets = [t(synth.targets(st.w.cfg, self.n, it)) for it in range(self.SETS)]
        self.queries = [gs.Query.jitter(self.DIMS, u) for u in self.offsets]
        self.val = torch.empty(self.n, device=dev)
        self.inf = torch.empty(self.n, device=dev)
        self.gv = torch.empty(self.n, device=dev)
        self.gi = torch.empty(self.n, device=dev)
        self.terms = gs.alloc_loss_terms(dev)
        self.loss_work = gs.alloc_loss_work(self.n, dev)
        self.grads = gs.Grads.empty(ng, dev)
        self.raw_grads = gs.RawParams(torch.empty(ng, 3, device=dev), torch.empty(ng, device=dev),
                                      torch.empty(ng, device=dev))
        self.grid = gs.make_grid(cells)
        self.activate()
        probe = gs.build_index(self.gauss, self.grid, TAU)
        self.index = gs.Index(self.grid, ng, int(probe.n_pairs * 1.25) + 4096, dev)
        del probe
        self.sp = SidePlans(gs, torch, self.queries[0], self.grid, dev)
        self.plan = self.sp.plans[0]
        gs.gs_build_index(self.gauss, self.grid, TAU, self.index)
        self.work = gs.alloc_backward_work(self.index, self.queries[0], dev)
        self.it = 0
        torch.cuda.synchronize()

    def activate(self):
        self.gs.gs_activate(self.raw, self.CAP, self.gauss.scale, self.gauss.value, self.gauss.weight)

    def densify_bench(self, k):
        """Pruning and densification after a step (Sec. 4.2.1), as training
        runs it every 100 iterations: weights below 0.005 removed, the
        2^21 samples ranked, and a fifth of the count (52,428) added at the
        worst samples within a target count 20 % above the current one.
        Each call includes its read-back of the new count."""
        gs, st, torch = self.gs, self.st, self.torch
        ng = st.g_host.n
        kmax = ng // 5
        cur = gs.ParamSet(st.dg.mean, self.raw.log_scale, st.dg.rot, self.raw.value_logit, self.raw.weight_logit)
        out = gs.ParamSet.empty(ng + kmax, "cuda:0")
        src = torch.empty(ng + kmax, dtype=torch.int32, device="cuda:0")
        q = self.queries[(self.it - 1) % self.SETS]
        work = gs.alloc_densify_work(ng, q, "cuda:0")
        tgt = self.targets[(self.it - 1) % self.SETS]

        def call():
            return gs.gs_densify(cur, ng, self.gauss.weight, self.grid, q, self.val, self.inf, tgt, None, 0.005, TAU,
                                 math.log(0.005), math.log(0.01 / 0.99), kmax, out, src, work)

        n_out = call()
        gs.profile_select(None)
        gs.profile_reset()
        gs.profile_enable(True)
        for _ in range(k):
            call()
        torch.cuda.synchronize()
        gs.profile_enable(False)
        kern = {name: round(ms / k * 1e3, 2) for name, (c, ms) in gs.profile_read().items()}
        t = timed(call, k, torch.cuda.synchronize)
        return {"ms_per_call": t * 1e3, "n_in": ng, "n_out": n_out, "added": n_out - int(src[:n_out].ge(0).sum()),
                "samples_ranked": self.n, "kernels_us": kern,
                "amortised_ms_per_step": t * 1e3 / 100.0}

    def step(self):
        gs, st = self.gs, self.st
        q = self.queries[self.it % self.SETS]
        # the query ordering on the side stream while activations and the
        # index build run (SidePlans)
        self.plan = self.sp.start(q, self.grid)
        self.activate()
        gs.gs_build_index(self.gauss, self.grid, TAU, self.index)
        self.sp.wait()
        gs.gs_sample_planned(self.gauss, self.index, q, self.val, self.inf, self.plan)
        gs.gs_loss(self.val, self.inf, self.targets[self.it % self.SETS], None, TAU, self.FN_EPS, self.FN_LAMBDA,
                   self.FP_LAMBDA, self.gv, self.gi, self.terms, self.loss_work)
        gs.gs_sample_backward(self.gauss, self.index, q, self.plan, self.val, self.inf, self.gv, self.gi, self.grads,
                              self.work)
        gs.gs_activate_backward(self.raw, self.CAP, self.grads, self.raw_grads)
        self.sp.release()
        self.it += 1


class ABStep:
    """Point-major (gs_sample) against Gaussian-major
    (gs_sample_gaussian_major, the paper's unstructured design) forward on a
    point-cloud workload: both whole calls, query ordering included, on the
    same index and points resident in HBM."""

    def __init__(self, name, batch_only):
        import numpy as np
        import torch

        import paper_2607_01164_amd as gs
        import synth
        self.gs, self.torch = gs, torch
        w = synth.WORKLOADS[name]
        self.w = w
        g = synth.make_gaussians(w)
        pts = synth.make_points(w)
        if batch_only:
            pts = pts[synth.batch_permutation(w, len(pts))[: w.batch]]
        self.n, self.n_gauss = len(pts), g.n
        dev = "cuda:0"
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        self.dg = gs.Gaussians(t(g.mean), t(g.scale), t(g.rot), t(g.value), t(g.weight))
        self.pts = t(pts)
        del pts
        self.grid = gs.make_grid(w.index_cells)
        self.index = gs.build_index(self.dg, self.grid, TAU)
        self.query = gs.Query.pts(self.pts)
        self.plan = gs.alloc_plan(self.query, self.grid, dev)
        self.work = gs.alloc_gaussian_major_work(self.query, dev)
        self.val = torch.empty(self.n, device=dev)
        self.inf = torch.empty(self.n, device=dev)
        torch.cuda.synchronize()

    def pm(self):
        self.gs.gs_sample(self.dg, self.index, self.query, self.val, self.inf, self.plan)

    def gm(self):
        self.gs.gs_sample_gaussian_major(self.dg, self.index, self.query, self.val, self.inf, self.plan, self.work)

    def run(self, k):
        gs, sync = self.gs, self.torch.cuda.synchronize
        out = {"workload": f"{self.w.name}: {self.n} points, {self.n_gauss} Gaussians, index "
                           f"{'x'.join(map(str, self.w.index_cells))} cells, forward only",
               "points": self.n}
        for name, fn in (("point_major", self.pm), ("gaussian_major", self.gm)):
            fn()
            sync()
            gs.profile_select(None)
            gs.profile_reset()
            gs.profile_enable(True)
            for _ in range(k):
                fn()
            sync()
            gs.profile_enable(False)
            kern = {kn: round(ms / k * 1e3, 1) for kn, (c, ms) in gs.profile_read().items()}
            t = timed(fn, k, sync)
            out[name] = {"ms": t * 1e3, "points_per_s": self.n / t, "kernels_us": kern}
        out["gaussian_major_over_point_major"] = out["gaussian_major"]["ms"] / out["point_major"]["ms"]
        return out


class ConfigStep:
    """One of the other workloads at its own configuration (index cells,
    queries), with the same calls as the headline step: index build,
    forward, and the backward where the workload has one. Inputs resident
    in HBM; each part timed over k calls."""

    def __init__(self, name):
        import numpy as np
        import torch

        import paper_2607_01164_amd as gs
        import synth
        self.gs, self.torch = gs, torch
        w = synth.WORKLOADS[name]
        self.w = w
        g = synth.make_gaussians(w)
        dev = "cuda:0"
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        self.dg = gs.Gaussians(t(g.mean), t(g.scale), t(g.rot), t(g.value), t(g.weight))
        self.grid = gs.make_grid(w.index_cells)
        if w.kind == "grid":
            self.query = gs.Query.grid(w.dims)
            self.plan = None
        else:
            pts = synth.make_points(w)
            if 0 < w.batch < len(pts):
                pts = pts[synth.batch_permutation(w, len(pts))[: w.batch]]
            self.pts = t(pts)
            del pts
            self.query = gs.Query.pts(self.pts)
            self.plan = gs.alloc_plan(self.query, self.grid, dev)
        self.n = self.query.size()
        probe = gs.build_index(self.dg, self.grid, TAU)
        self.index = gs.Index(self.grid, g.n, int(probe.n_pairs * 1.25) + 4096, dev)
        del probe
        gs.gs_build_index(self.dg, self.grid, TAU, self.index)
        self.val = torch.empty(self.n, device=dev)
        self.inf = torch.empty(self.n, device=dev)
        self.has_bwd = w.backward
        if self.has_bwd:
            gv, gi = synth.cotangents(w, self.n)
            self.gv, self.gi = t(gv), t(gi)
            self.grads = gs.Grads.empty(g.n, dev)
            self.work = gs.alloc_backward_work(self.index, self.query, dev)
        torch.cuda.synchronize()

    def build(self):
        self.gs.gs_build_index(self.dg, self.grid, TAU, self.index)

    def forward(self):
        self.gs.gs_sample(self.dg, self.index, self.query, self.val, self.inf, self.plan)

    def backward(self):
        self.gs.gs_sample_backward(self.dg, self.index, self.query, self.plan, self.val, self.inf, self.gv, self.gi,
                                   self.grads, self.work)

    def run(self, k, tag):
        gs, sync = self.gs, self.torch.cuda.synchronize
        self.build()
        self.forward()
        if self.has_bwd:
            self.backward()
        sync()
        tb = timed(self.build, k, sync)
        fk = "sample_grid" if self.w.kind == "grid" else "sample_points"
        tf, fwd_us, _ = kernel_avg_us(gs, fk, self.forward, k, sync)
        work = self.work if self.has_bwd else gs.alloc_backward_work(self.index, self.query, "cuda:0")
        self.forward()
        tests, contrib = gs.sample_pair_counts(self.index, self.query, self.plan, work)
        out = {"workload": self.w.description, "queries": self.n, "index_cells": list(self.w.index_cells),
               "index_pairs": self.index.n_pairs, "ms_build": tb * 1e3, "ms_fwd": tf * 1e3,
               "fwd_points_per_s": self.n / tf, "forward_tests": tests, "contributing_pairs": contrib,
               "gauss_point_evals_per_s": contrib / tf,
               "samplers": {fk: sampler_entry(fk, tag, fwd_us, tests, contrib)}}
        if self.has_bwd:
            self.forward()
            tw, bwd_us, _ = kernel_avg_us(gs, "bwd_gauss", self.backward, k, sync)
            bt = gs.backward_pair_count(self.index, self.query, self.plan, self.work)
            out.update({"ms_bwd": tw * 1e3, "fwd_bwd_samples_per_s": self.n / (tb + tf + tw),
                        "fwd_bwd_samples_per_s_excl_build": self.n / (tf + tw), "backward_tests": bt})
            out["samplers"]["bwd_gauss"] = sampler_entry("bwd_gauss", tag, bwd_us, bt, contrib)
        return out


def sampler_flops(kernel, tests, contrib):
    """Algorithmic flops of one sampler launch from its tested and
    contributing pairs."""
    return FLOPS_FAILING_PAIR * (tests - contrib) + FLOPS_CONTRIB[kernel] * contrib


def sampler_entry(kernel, tag, avg_us, tests, contrib):
    """A sampler kernel's algorithmic rate against the fp32 vector peak, and
    its HBM traffic (committed counter reading, when the sources match)
    against the HBM peak."""
    out = {"avg_us": avg_us, "pair_tests": tests, "contributing_pairs": contrib}
    if avg_us:
        fl = sampler_flops(kernel, tests, contrib)
        out.update({"flops_per_launch": fl, "tflops": fl / (avg_us * 1e-6) / 1e12,
                    "frac": fl / (avg_us * 1e-6) / 1e12 / FP32_VEC_PEAK_TFLOPS})
    tr = measured_traffic(kernel, tag)
    out["hbm_bytes"] = tr
    out["hbm_frac"] = (tr / (avg_us * 1e-6) / (HBM_PEAK_GBS * 1e9)) if (tr and avg_us) else None
    return out


def cpu_baseline(st: PointsStep, target_s: float):
    """The oracle (float64 brute force over every Gaussian, OpenMP over
    points, then Gaussian-major backward) on a seeded sample of the first
    batch."""
    import numpy as np

    import oracle
    g = st.g_host
    sel_all = np.random.default_rng(11).permutation(st.n)
    threads = oracle.default_threads()
    gv_all, gi_all = st.gv[0].cpu().numpy(), st.gi[0].cpu().numpy()

    def run(m):
        sel = sel_all[:m]
        pts = st.batch0_host[sel]
        t0 = time.perf_counter()
        ref = oracle.forward(g, pts, tau=TAU, threads=threads)
        oracle.backward(g, pts, ref.phi, ref.inf, gv_all[sel], gi_all[sel], tau=TAU, threads=threads)
        return time.perf_counter() - t0, ref

    m = 256
    dt, ref = run(m)
    m2 = int(min(65536, max(m, m * target_s / max(dt, 1e-3))))
    if m2 > m:
        dt, ref = run(m2)
        m = m2
    return {"value": m / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
            "sample": f"{m} of the {st.n} points of the first batch, forward + backward to all {g.n} Gaussians, "
                      f"{dt:.1f} s"}


def run_only(a):
    """One workload's step loop alone (warmup + steps), for profiling."""
    import torch
    sync = torch.cuda.synchronize
    if a.only == "c4":
        st = PointsStep(HEADLINE)
        fn, n = st.step, st.n * st.batches
    elif a.only == "c2":
        st = GridBatchStep()
        fn, n = st.step, st.n
    elif a.only == "train":
        ts = TrainStep(GridBatchStep(), TRAIN_CELLS)
        fn, n = ts.step, ts.n
    else:
        name = {"c5": "c5_points100m", "c3": "c3_grid512_full", "c1": "c1_grid32"}[a.only]
        cs = ConfigStep(name)

        def fn():
            cs.build()
            cs.forward()
            if cs.has_bwd:
                cs.backward()
        n = cs.n
    import paper_2607_01164_amd as gs
    for _ in range(a.warmup):
        fn()
    sync()
    t = timed(fn, a.steps, sync)
    kern = {k: round(v[1], 2) for k, v in kernel_table(gs, fn, a.steps, sync).items()}
    print(json.dumps({"only": a.only, "steps": a.steps, "ms_per_step": t * 1e3, "per_s": n / t, "kernels_us": kern}),
          flush=True)
    if a.copy_probe:
        copy_probe()


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); the sharded path is not built",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2607_01164_amd as gs
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if a.only:
        run_only(a)
        return
    sync = torch.cuda.synchronize
    st = PointsStep(HEADLINE)
    for _ in range(a.warmup):
        st.step()
    sync()
    # untimed pass with every kernel bracketed by events: the per-kernel table
    # and the dominant kernel
    kernels = kernel_table(gs, st.step, a.steps, sync)
    dom = max(kernels.items(), key=lambda kv: kv[1][1])[0]
    # timed region: K whole steps; only the dominant kernel is bracketed by
    # HIP events (on the library's stream), for its roofline entry
    t_step, dom_us, dom_launches = kernel_avg_us(gs, dom, st.step, a.steps, sync)
    counts = st.pair_counts()
    tests = sum(c[0] for c in counts) / len(counts)
    btests = sum(c[1] for c in counts) / len(counts)
    contrib = sum(c[2] for c in counts) / len(counts)
    # the parts alone, per batch, for the query rates
    t_build = timed(st.build, a.steps, sync)
    st.b = 0
    t_fwd, fwd_us, _ = kernel_avg_us(gs, "sample_points", lambda: st.forward(0), a.steps, sync)
    t_bwd, bwd_us, _ = kernel_avg_us(gs, "bwd_gauss", lambda: st.backward(0), a.steps, sync)
    samplers = {"sample_points": sampler_entry("sample_points", HEADLINE, fwd_us, tests, contrib),
                "bwd_gauss": sampler_entry("bwd_gauss", HEADLINE, bwd_us, btests, contrib)}
    roof = roofline(dom, dom_us, dom_launches, tests, btests, contrib, st.index.n_pairs)
    n_step = st.n * st.batches

    c5 = None
    if not a.no_c5:
        cs = ConfigStep("c5_points100m")
        c5 = cs.run(3, "c5_points100m")
        del cs
        torch.cuda.empty_cache()
    extras = {}
    if not a.no_extras:
        c2 = GridBatchStep()
        for _ in range(a.warmup):
            c2.step()
        t2 = timed(c2.step, a.steps, sync)
        t2f, f2_us, _ = kernel_avg_us(gs, "sample_points", c2.forward, a.steps, sync)
        t2b, b2_us, _ = kernel_avg_us(gs, "bwd_gauss", c2.backward, a.steps, sync)
        t2i = timed(c2.build, a.steps, sync)
        ct, cbt, cc = c2.pair_counts()
        extras["c2_grid256_batch"] = {
            "workload": f"structured 256^3 grid, 262144 Gaussians, batch of 2^20 random voxel centres, index "
                        f"{'x'.join(map(str, c2.cells))} cells, step = build + forward + backward",
            "samples_per_step": c2.n, "ms_per_step": t2 * 1e3, "fwd_bwd_samples_per_s": c2.n / t2,
            "ms_build": t2i * 1e3, "ms_fwd": t2f * 1e3, "ms_bwd": t2b * 1e3, "index_pairs": c2.index.n_pairs,
            "forward_tests": ct, "backward_tests": cbt, "contributing_pairs": cc,
            "gauss_point_evals_per_s": cc / t2f,
            "samplers": {"sample_points": sampler_entry("sample_points", "c2_grid256_batch", f2_us, ct, cc),
                         "bwd_gauss": sampler_entry("bwd_gauss", "c2_grid256_batch", b2_us, cbt, cc)},
            "kernels_us": {k: round(v[1], 2) for k, v in kernel_table(gs, c2.step, a.steps, sync).items()}}
        ts = TrainStep(c2, TRAIN_CELLS)
        for _ in range(a.warmup):
            ts.step()
        sync()
        tk = {k: round(v[1], 2) for k, v in kernel_table(gs, ts.step, a.steps, sync).items()}
        t_ts = timed(ts.step, a.steps, sync)
        terms = gs.read_loss_terms(ts.terms)
        dens = ts.densify_bench(a.steps)
        extras["training_step"] = {
            "workload": "structured training step: free parameters of the 262144 Gaussians -> activations "
                        f"(soft norm cap 0.02) -> index ({'x'.join(map(str, TRAIN_CELLS))} cells) -> 128^3 "
                        "jittered samples (one random position per "
                        f"voxel, offsets and targets redrawn each step from {TrainStep.SETS} sets resident in "
                        "HBM) -> forward -> L1 + false-negative losses -> backward -> activation backward",
            "samples_per_step": ts.n, "ms_per_step": t_ts * 1e3, "fwd_bwd_samples_per_s": ts.n / t_ts,
            "loss": {k: terms[k] for k in ("l1", "fn", "total", "n_fn")}, "kernels_us": tk, "densify": dens}
        del ts, c2
        torch.cuda.empty_cache()
        for name in ("c1_grid32", "c3_grid512_full"):
            cs = ConfigStep(name)
            extras[name] = cs.run(3 if cs.n > 5e7 else a.steps, name)
            del cs
            torch.cuda.empty_cache()
        extras["forward_ab_c4"] = ABStep("c4_points8m", True).run(max(3, a.steps // 3))
        sync()
    if a.breakdown:
        for k, (c, us) in sorted(kernels.items(), key=lambda kv: -kv[1][1]):
            log(f"{k:18s} {us:9.1f} us/step  {c:5.1f} launches")
    if a.copy_probe:
        copy_probe()

    cpu = None if a.no_cpu else cpu_baseline(st, a.cpu_seconds)
    out = {
        "metric": "query points/sec fwd and fwd+bwd samples/sec; % of HBM roofline",
        "value": n_step / t_step,
        "unit": "fwd+bwd samples/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{HEADLINE}: 8388608 clustered points (64-component anisotropic mixture, cavity of "
                               f"radius 0.2), {st.g_host.n} Gaussians, index "
                               f"{'x'.join(map(str, st.w.index_cells))} cells; step = {st.batches} batches of "
                               f"{st.n} points, each build + forward + backward",
                   "global_batch": n_step, "batch": st.n, "batches": st.batches, "n_gauss": st.g_host.n,
                   "index_pairs": st.index.n_pairs, "forward_tests": tests, "backward_tests": btests,
                   "contributing_pairs": contrib},
        "fwd_points_per_s": st.n / t_fwd,
        "fwd_bwd_samples_per_s_excl_build": st.n / (t_fwd + t_bwd),
        "ms_build": t_build * 1e3, "ms_fwd": t_fwd * 1e3, "ms_bwd": t_bwd * 1e3,
        "gauss_point_evals_per_s": contrib / t_fwd,
        "samplers": samplers,
        "kernels": {k: round(v[1], 2) for k, v in kernels.items()},
        "roofline": roof,
        "c5_points100m_forward": c5,
        "secondary": extras or None,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def copy_probe():
    """A plain device copy of COPY_PROBE_BYTES (read once, written once), so
    that a counter run sees the HBM bytes of a kernel of known traffic."""
    import torch
    src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()


def source_digest():
    """sha256 over the kernel sources; a stored counter reading is used only
    while the sources it was taken on are unchanged."""
    h = hashlib.sha256()
    for f in sorted(os.listdir(SRC_DIR)):
        if f.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(SRC_DIR, f), "rb") as fh:
                h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    counter summary (FETCH_SIZE + WRITE_SIZE, scaled by the copy-probe
    calibration), or None when there is none or the kernel sources changed
    since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    dig = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not dig or not val or dig.group(1) != source_digest():
        return None
    return float(val.group(1))


def roofline(name, avg_us, launches, tests, btests, contrib, n_pairs):
    """Roofline entry of the dominant kernel: algorithmic flops (or bytes) of
    one launch over its average launch duration (HIP events on the stream the
    kernel runs on, over the timed region)."""
    avg_s = avg_us * 1e-6
    out = {"kernel": name, "avg_us": avg_us, "launches_per_step": launches}
    traffic = measured_traffic(name, HEADLINE)
    if name in FLOPS_CONTRIB:
        t = btests if name == "bwd_gauss" else tests
        flops = sampler_flops(name, t, contrib)
        ach = flops / avg_s / 1e12
        out.update({"bound": "alu", "achieved": ach, "peak": FP32_VEC_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": ach / FP32_VEC_PEAK_TFLOPS, "traffic": traffic, "flops_per_launch": flops,
                    "pair_tests": t, "contributing_pairs": contrib,
                    "hbm_frac": (traffic / avg_s / (HBM_PEAK_GBS * 1e9)) if traffic else None})
        return out
    per_pair = {"radix_downsweep": SORT_BYTES_PER_PAIR, "emit": EMIT_BYTES_PER_PAIR}.get(name)
    if per_pair is None:
        out.update({"bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": None,
                    "traffic": traffic})
        return out
    byts = per_pair * n_pairs
    ach = byts / avg_s / 1e9
    out.update({"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
                "traffic": traffic, "bytes_per_launch": byts})
    return out


if __name__ == "__main__":
    main()
