"""Benchmark of the Gaussian-field sampling hot path on one MI355X.

Workload: structured 256^3 grid over [0,1]^3, 262,144 Gaussians (means
U[0,1]^3, log-scales N(ln 0.008, 0.4) per axis, random unit quaternions,
values U[0,1], weights sigmoid(N(0,1))); one step is a training step on a
seeded random batch of 2^20 voxel centres: build the cell index, sample
(query ordering + forward) and backpropagate N(0,1) cotangents to every
Gaussian parameter. All inputs are resident in HBM before the timed region.

Prints one JSON line: fwd+bwd samples/s over the timed steps, with the
forward-only query rate, the per-kernel timing of the step (HIP events on
the library's stream), the roofline of the dominant kernel, the CPU
oracle's rate on a bounded sample of the same workload, and the rate of a
structured training step: activations, index, 128^3 jittered samples (one
random position per voxel), losses, backward and the activations' backward
over the free parameters behind the same Gaussians.
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
# Algorithmic work, counted as adds and multiplies (an FMA is 2) and the
# exponential as 1. Every candidate (Gaussian, point) pair of a cell list is
# tested: d = p - mu (3), u = M d (15), Q = |u|^2 (5), the cutoff compare (1).
# A contributing pair (Q <= T) adds, in the forward, a = w exp(-Q/2),
# I += a, V += a v; in the backward, a, dL/da, the per-pair moment terms and
# dv, dw.
FLOPS_PER_TEST = 24.0
FLOPS_PER_CONTRIB = {"sample_points": 7.0, "sample_grid": 7.0, "bwd_gauss": 37.0}
# Bytes one pass of the LSD sort moves per pair: read and write key and value.
SORT_BYTES_PER_PAIR = 16.0
EMIT_BYTES_PER_PAIR = 8.0
COPY_PROBE_BYTES = 256 << 20   # plain copy used to calibrate the HBM byte counters
SRC_DIR = os.path.join(ROOT, "paper_2607_01164_amd", "csrc")
WORKLOAD = "c2_grid256_batch"
INDEX_CELLS = (32, 32, 32)
TRAIN_CELLS = (40, 40, 40)     # the training step's index: twice C2's query density
TAU = 0.01


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--cells", type=int, nargs=3, default=list(INDEX_CELLS))
    p.add_argument("--train-cells", type=int, nargs=3, default=list(TRAIN_CELLS))
    p.add_argument("--cpu-seconds", type=float, default=16.0, help="target length of the CPU oracle sample")
    p.add_argument("--no-cpu", action="store_true")
    p.add_argument("--no-train", action="store_true", help="skip the 128^3 structured training-step line")
    p.add_argument("--no-ab", action="store_true", help="skip the point-major / Gaussian-major comparison")
    p.add_argument("--ab-c5", action="store_true",
                   help="also compare the two forwards on the 10^8-point cloud (slow to generate)")
    p.add_argument("--no-configs", action="store_true", help="skip the C1, C3 and C4 lines")
    p.add_argument("--breakdown", action="store_true", help="print the per-kernel table to stderr")
    p.add_argument("--copy-probe", action="store_true",
                   help="after the timed region, run a plain 256 MiB copy (counter calibration under rocprofv3)")
    return p.parse_args()


class Step:
    def __init__(self, cells):
        import numpy as np
        import torch

        import paper_2607_01164_amd as gs
        import synth
        self.gs, self.torch, self.np = gs, torch, np
        w = synth.WORKLOADS[WORKLOAD]
        self.w = w
        g = synth.make_gaussians(w)
        self.g_host = g
        self.ids_host = synth.voxel_batch(w)
        gv, gi = synth.cotangents(w, len(self.ids_host))
        dev = "cuda:0"
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        self.dg = gs.Gaussians(t(g.mean), t(g.scale), t(g.rot), t(g.value), t(g.weight))
        self.ids = torch.from_numpy(self.ids_host.view(np.int32)).to(dev)
        self.gv, self.gi = t(gv), t(gi)
        self.grid = gs.make_grid(cells)
        self.query = gs.Query.voxels(w.dims, self.ids)
        self.n = len(self.ids_host)
        probe = gs.build_index(self.dg, self.grid, TAU)
        self.index = gs.Index(self.grid, g.n, int(probe.n_pairs * 1.25) + 4096, dev)
        del probe
        self.plan = gs.alloc_plan(self.query, self.grid, dev)
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
        self.build()
        self.forward()
        self.backward()

    def candidate_tests(self) -> int:
        """(Gaussian, point) pairs the forward and the backward test: the sum
        over cells of (pairs listed in the cell) x (queries in the cell), from
        the index's cell offsets and the plan's per-cell query offsets (after
        the four 256-byte aligned query-length arrays of the plan, one offset
        per quarter of a cell along x)."""
        torch = self.torch
        ncells = self.grid.cells[0] * self.grid.cells[1] * self.grid.cells[2]
        al = lambda b: (b + 255) // 256 * 256
        off = 4 * al(4 * max(self.n, 1))
        # the plan's offsets are per quarter of a cell along x (4 keys a cell)
        point_off = self.plan[off: off + 4 * (4 * ncells + 2)].view(torch.int32).to(torch.int64)
        pts = point_off[4:4 * ncells + 1:4] - point_off[0:4 * ncells:4]
        co = self.index.cell_offsets.to(torch.int64)
        pairs = co[1:] - co[:-1]
        return int((pts * pairs).sum().item())


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

    def __init__(self, st: Step, cells):
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
        self.plan = gs.alloc_plan(self.queries[0], self.grid, dev)
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
        self.activate()
        gs.gs_build_index(self.gauss, self.grid, TAU, self.index)
        gs.gs_sample(self.gauss, self.index, q, self.val, self.inf, self.plan)
        gs.gs_loss(self.val, self.inf, self.targets[self.it % self.SETS], None, TAU, self.FN_EPS, self.FN_LAMBDA,
                   self.FP_LAMBDA, self.gv, self.gi, self.terms, self.loss_work)
        gs.gs_sample_backward(self.gauss, self.index, q, self.plan, self.val, self.inf, self.gv, self.gi, self.grads,
                              self.work)
        gs.gs_activate_backward(self.raw, self.CAP, self.grads, self.raw_grads)
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

    def run(self, k):
        sync = self.torch.cuda.synchronize
        self.build()
        self.forward()
        if self.has_bwd:
            self.backward()
        sync()
        tb, tf = timed(self.build, k, sync), timed(self.forward, k, sync)
        out = {"workload": self.w.description, "queries": self.n, "index_cells": list(self.w.index_cells),
               "index_pairs": self.index.n_pairs, "ms_build": tb * 1e3, "ms_fwd": tf * 1e3,
               "fwd_points_per_s": self.n / tf}
        if self.has_bwd:
            self.forward()
            tw = timed(self.backward, k, sync)
            out.update({"ms_bwd": tw * 1e3, "fwd_bwd_samples_per_s": self.n / (tb + tf + tw),
                        "fwd_bwd_samples_per_s_excl_build": self.n / (tf + tw)})
        return out


def timed(fn, k, sync):
    sync()
    t0 = time.perf_counter()
    for _ in range(k):
        fn()
    sync()
    return (time.perf_counter() - t0) / k


def cpu_baseline(st: Step, target_s: float):
    """The oracle (float64 brute force over every Gaussian, OpenMP over
    points, then Gaussian-major backward) on a seeded sample of the batch."""
    import numpy as np

    import oracle
    g = st.g_host
    sel_all = np.random.default_rng(11).permutation(st.n)
    threads = oracle.default_threads()

    def run(m):
        sel = sel_all[:m]
        pts = oracle.voxel_centers(st.w.dims, ids=st.ids_host[sel])
        gv = st.gv.cpu().numpy()[sel]
        gi = st.gi.cpu().numpy()[sel]
        t0 = time.perf_counter()
        ref = oracle.forward(g, pts, tau=TAU, threads=threads)
        oracle.backward(g, pts, ref.phi, ref.inf, gv, gi, tau=TAU, threads=threads)
        return time.perf_counter() - t0, ref

    m = 512
    dt, ref = run(m)
    m2 = int(min(65536, max(m, m * target_s / max(dt, 1e-3))))
    if m2 > m:
        dt, ref = run(m2)
        m = m2
    return {"value": m / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
            "sample": f"{m} of the {st.n} batch voxels, forward + backward to all {g.n} Gaussians, {dt:.1f} s",
            "contrib_per_point": float(ref.ncontrib.mean())}


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); the sharded path is not built",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2607_01164_amd as gs
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    st = Step(tuple(a.cells))
    sync = torch.cuda.synchronize
    for _ in range(a.warmup):
        st.step()
    sync()
    # untimed pass with every kernel bracketed by events: the per-kernel table
    # and the dominant kernel
    gs.profile_select(None)
    gs.profile_reset()
    gs.profile_enable(True)
    for _ in range(a.steps):
        st.step()
    sync()
    gs.profile_enable(False)
    prof = gs.profile_read()
    kernels = {k: {"launches_per_step": c / a.steps, "ms_per_step": ms / a.steps, "avg_ms": ms / c}
               for k, (c, ms) in prof.items()}
    dom_name = max(kernels.items(), key=lambda kv: kv[1]["ms_per_step"])[0]
    # timed region: K whole steps; only the dominant kernel is bracketed by
    # HIP events (on the library's stream), for its roofline entry
    gs.profile_select(dom_name)
    gs.profile_reset()
    gs.profile_enable(True)
    t_step = timed(st.step, a.steps, sync)
    gs.profile_enable(False)
    gs.profile_select(None)
    c, ms = gs.profile_read()[dom_name]
    dom = (dom_name, {"launches_per_step": c / a.steps, "ms_per_step": ms / a.steps, "avg_ms": ms / c})
    n_pairs = st.index.n_pairs
    n_tests = st.candidate_tests()
    bwd_tests = gs.backward_pair_count(st.index, st.query, st.plan, st.work)
    # forward alone and backward alone, for the query rates
    t_fwd = timed(st.forward, a.steps, sync)
    t_bwd = timed(st.backward, a.steps, sync)
    t_build = timed(st.build, a.steps, sync)
    train = None
    if not a.no_train:
        ts = TrainStep(st, tuple(a.train_cells))
        for _ in range(a.warmup):
            ts.step()
        sync()
        gs.profile_select(None)
        gs.profile_reset()
        gs.profile_enable(True)
        for _ in range(a.steps):
            ts.step()
        sync()
        gs.profile_enable(False)
        tk = {k: round(ms / a.steps * 1e3, 2) for k, (c, ms) in gs.profile_read().items()}
        t_ts = timed(ts.step, a.steps, sync)
        terms = gs.read_loss_terms(ts.terms)
        dens = ts.densify_bench(a.steps)
        train = {"workload": "structured training step: free parameters of the 262144 Gaussians -> activations "
                             f"(soft norm cap 0.02) -> index ({'x'.join(map(str, a.train_cells))} cells) -> 128^3 "
                             "jittered samples (one random position per "
                             f"voxel, offsets and targets redrawn each step from {TrainStep.SETS} sets resident in "
                             "HBM) -> forward -> L1 + false-negative losses -> backward -> activation backward",
                 "samples_per_step": ts.n, "ms_per_step": t_ts * 1e3, "fwd_bwd_samples_per_s": ts.n / t_ts,
                 "loss": {k: terms[k] for k in ("l1", "fn", "total", "n_fn")}, "kernels_us": tk,
                 "densify": dens}
        del ts

    configs = None
    if not a.no_configs:
        configs = {}
        for name in ("c1_grid32", "c3_grid512_full", "c4_points8m") + (("c5_points100m",) if a.ab_c5 else ()):
            cs = ConfigStep(name)
            configs[name] = cs.run(3 if cs.n > 5e7 else max(5, a.steps // 5))
            del cs
            torch.cuda.empty_cache()
    ab = None
    if not a.no_ab:
        ab = {"c4": ABStep("c4_points8m", True).run(max(3, a.steps // 5))}
        if a.ab_c5:
            ab["c5"] = ABStep("c5_points100m", False).run(3)
        sync()
    if a.breakdown:
        for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
            log(f"{k:18s} {v['ms_per_step'] * 1e3:9.1f} us/step  {v['launches_per_step']:5.1f} launches  "
                f"avg {v['avg_ms'] * 1e3:9.1f} us")
    if a.copy_probe:
        copy_probe()

    cpu = None if a.no_cpu else cpu_baseline(st, a.cpu_seconds)
    contrib = cpu.pop("contrib_per_point") if cpu else None
    roof = roofline(dom[0], dom[1], st, n_pairs, bwd_tests if dom[0] == "bwd_gauss" else n_tests, contrib)
    out = {
        "metric": "query points/sec fwd and fwd+bwd samples/sec; % of HBM roofline",
        "value": st.n / t_step,
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
        "config": {"workload": f"{WORKLOAD}: 256^3 grid, 262144 Gaussians, batch of 2^20 random voxel centres, "
                               f"index {a.cells[0]}x{a.cells[1]}x{a.cells[2]} cells, step = build + forward + backward",
                   "global_batch": st.n, "n_gauss": st.g_host.n, "index_pairs": n_pairs,
                   "candidate_tests": n_tests, "backward_tests": bwd_tests},
        "fwd_points_per_s": st.n / t_fwd,
        "fwd_bwd_samples_per_s_excl_build": st.n / (t_fwd + t_bwd),
        "ms_build": t_build * 1e3, "ms_fwd": t_fwd * 1e3, "ms_bwd": t_bwd * 1e3,
        "gauss_point_evals_per_s": (contrib * st.n / t_fwd) if contrib else None,
        "candidate_tests_per_s_fwd": n_tests / t_fwd,
        "candidate_tests_per_s_bwd": bwd_tests / t_bwd,
        "kernels": {k: round(v["ms_per_step"] * 1e3, 2) for k, v in kernels.items()},
        "training_step": train,
        "forward_ab": ab,
        "configs": configs,
        "roofline": roof,
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


def measured_traffic(name):
    """HBM bytes per launch of kernel `name` from the committed counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by the copy-probe calibration),
    or None when there is none or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", f"{name}_c2_step_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    dig = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not dig or not val or dig.group(1) != source_digest():
        return None
    return float(val.group(1))


def roofline(name, k, st, n_pairs, n_tests, contrib_per_point):
    """Roofline entry of the dominant kernel: algorithmic flops (or bytes) of
    one launch over its average launch duration (HIP events on the stream the
    kernel runs on)."""
    avg_s = k["avg_ms"] * 1e-3
    out = {"kernel": name, "avg_us": avg_s * 1e6, "launches_per_step": k["launches_per_step"]}
    traffic = measured_traffic(name)
    if name in FLOPS_PER_CONTRIB:
        # units: the pairs the launch tests (exact: for the forward, the cell
        # lists times the cells' queries, from the index and the plan; for the
        # backward, the queries of each Gaussian's trimmed rows, counted by
        # the library) and its contributing pairs (the oracle's count per
        # point on the CPU-baseline sample, times the batch; None without it)
        if contrib_per_point is None:
            out.update({"bound": "alu", "achieved": None, "peak": FP32_VEC_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": None, "traffic": traffic, "pair_tests": n_tests})
            return out
        units = contrib_per_point * st.n
        flops = FLOPS_PER_TEST * n_tests + FLOPS_PER_CONTRIB[name] * units
        ach = flops / avg_s / 1e12
        out.update({"bound": "alu", "achieved": ach, "peak": FP32_VEC_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": ach / FP32_VEC_PEAK_TFLOPS, "traffic": traffic,
                    "flops_per_launch": flops, "pair_tests": n_tests, "contributing_pairs": units})
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
