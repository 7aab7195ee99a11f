"""Seeded synthetic inputs for the Gaussian-field sampler.

This module draws random numbers and nothing else: Gaussian parameter sets,
query point clouds, query batches and cotangents. It holds none of the
sampling method's arithmetic, so the GPU library and the CPU oracle both
take their inputs from here without sharing any of the computation.

Every draw uses ``numpy.random.Generator(PCG64(SeedSequence(SEED,
spawn_key=(config, stream))))``; draws are made in float64 and rounded once
to float32. Streams: 0 means, 1 log-scales, 2 quaternions, 3 values,
4 weights, 5 mixture used for the means, 6 query points, 7 batch selection,
8 cotangents, 9 mixture components.

The five workloads stand in for the paper's datasets (Open SciVis structured
volumes, the unstructured meshes of its Appendix A), which are not available:
every domain is normalised to [0,1]^3 as the paper does in its structured
evaluation (Sec. 6.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np

SEED = 260701164

# stream ids
S_MEAN, S_LOGSCALE, S_QUAT, S_VALUE, S_WEIGHT, S_MEANMIX, S_POINTS, S_BATCH, S_COTAN, S_COMP, S_JITTER, S_TARGET = \
    range(12)


def rng(cfg: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(cfg, stream))))


@dataclass
class Mixture:
    """Anisotropic Gaussian-mixture point density on [0,1]^3 with optional
    spherical cavities. Rotations are Haar-random orthogonal matrices from a
    QR factorisation (not the sampler's quaternion convention)."""
    n_comp: int
    std_lo: float
    std_hi: float
    uniform_frac: float = 0.0
    cavities: Tuple[Tuple[Tuple[float, float, float], float], ...] = ()
    centers: Optional[np.ndarray] = None
    stds: Optional[np.ndarray] = None
    rots: Optional[np.ndarray] = None

    def build(self, g: np.random.Generator) -> "Mixture":
        self.centers = g.uniform(0.1, 0.9, size=(self.n_comp, 3))
        self.stds = np.exp(g.uniform(np.log(self.std_lo), np.log(self.std_hi), size=(self.n_comp, 3)))
        rots = np.empty((self.n_comp, 3, 3))
        for k in range(self.n_comp):
            a = g.standard_normal((3, 3))
            qm, rm = np.linalg.qr(a)
            qm = qm * np.sign(np.diag(rm))[None, :]
            if np.linalg.det(qm) < 0:
                qm[:, 0] = -qm[:, 0]
            rots[k] = qm
        self.rots = rots
        return self

    def _accept(self, x: np.ndarray) -> np.ndarray:
        ok = np.all((x >= 0.0) & (x <= 1.0), axis=1)
        for c, r in self.cavities:
            ok &= np.sum((x - np.asarray(c)[None, :]) ** 2, axis=1) >= r * r
        return ok

    def sample(self, g: np.random.Generator, n: int, dtype=np.float64) -> np.ndarray:
        """n accepted points, drawn in rounds of at most 2^22 candidates with
        rejection; stored as `dtype`."""
        out = np.empty((n, 3), dtype=dtype)
        filled = 0
        while filled < n:
            m = min(1 << 22, max(1024, int((n - filled) * 1.3)))
            is_uni = g.random(m) < self.uniform_frac
            comp = g.integers(0, self.n_comp, size=m)
            z = g.standard_normal((m, 3)) * self.stds[comp]
            x = self.centers[comp] + np.einsum("nij,nj->ni", self.rots[comp], z)
            u = g.random((m, 3))
            x = np.where(is_uni[:, None], u, x)
            x = x[self._accept(x)]
            take = min(len(x), n - filled)
            out[filled:filled + take] = x[:take]
            filled += take
        return out


@dataclass
class Gaussians:
    mean: np.ndarray    # [n,3] f32
    scale: np.ndarray   # [n,3] f32, post-activation standard deviations
    rot: np.ndarray     # [n,4] f32, (w,x,y,z)
    value: np.ndarray   # [n]   f32
    weight: np.ndarray  # [n]   f32

    @property
    def n(self) -> int:
        return int(self.mean.shape[0])

    def subset(self, idx) -> "Gaussians":
        return Gaussians(self.mean[idx], self.scale[idx], self.rot[idx], self.value[idx], self.weight[idx])


@dataclass
class Workload:
    name: str
    cfg: int
    n_gauss: int
    log_scale_mu: float
    log_scale_sd: float
    kind: str                      # "grid" | "voxels" | "points"
    dims: Tuple[int, int, int] = (0, 0, 0)
    index_cells: Tuple[int, int, int] = (0, 0, 0)
    batch: int = 0                 # query points per batch (voxels/points)
    n_points: int = 0              # point cloud size (points)
    backward: bool = True
    mean_mix: Optional[Mixture] = None
    mean_mix_frac: float = 0.0     # fraction of means drawn from the mixture
    point_mix: Optional[Mixture] = None
    lo: Tuple[float, float, float] = (0.0, 0.0, 0.0)
    hi: Tuple[float, float, float] = (1.0, 1.0, 1.0)
    description: str = ""


def _c3_mix():
    return Mixture(n_comp=32, std_lo=0.02, std_hi=0.08)


def _c4_mix():
    return Mixture(n_comp=64, std_lo=0.01, std_hi=0.1, cavities=(((0.5, 0.5, 0.5), 0.2),))


def _c5_mix():
    return Mixture(n_comp=256, std_lo=0.002, std_hi=0.05, uniform_frac=0.3,
                   cavities=(((0.3, 0.3, 0.3), 0.15), ((0.7, 0.7, 0.7), 0.15)))


WORKLOADS = {
    "c1_grid32": Workload(
        name="c1_grid32", cfg=0, n_gauss=4096, log_scale_mu=np.log(0.03), log_scale_sd=0.3,
        kind="grid", dims=(32, 32, 32), index_cells=(8, 8, 8),
        description="structured 32^3 grid, all voxel centers, 4,096 Gaussians, fwd+bwd"),
    "c2_grid256_batch": Workload(
        name="c2_grid256_batch", cfg=1, n_gauss=262144, log_scale_mu=np.log(0.008), log_scale_sd=0.4,
        kind="voxels", dims=(256, 256, 256), index_cells=(64, 64, 64), batch=1 << 20,
        description="structured 256^3 grid, 262,144 Gaussians, fwd+bwd on a random batch of 2^20 voxel centers"),
    "c3_grid512_full": Workload(
        name="c3_grid512_full", cfg=2, n_gauss=1048576, log_scale_mu=np.log(0.004), log_scale_sd=0.5,
        kind="grid", dims=(512, 512, 512), index_cells=(128, 128, 128), backward=False,
        mean_mix_frac=0.7,
        description="structured 512^3 full-volume forward, 1,048,576 Gaussians (70% clustered means)"),
    "c4_points8m": Workload(
        name="c4_points8m", cfg=3, n_gauss=524288, log_scale_mu=np.log(0.005), log_scale_sd=0.8,
        kind="points", index_cells=(64, 64, 64), batch=1 << 21, n_points=8388608,
        mean_mix_frac=1.0,
        description="unstructured 8M clustered points with a cavity, 524,288 Gaussians, fwd+bwd on 2^21-point batches"),
    "c5_points100m": Workload(
        name="c5_points100m", cfg=4, n_gauss=2097152, log_scale_mu=np.log(0.003), log_scale_sd=1.0,
        kind="points", index_cells=(64, 64, 64), batch=100_000_000, n_points=100_000_000, backward=False,
        mean_mix_frac=1.0,
        description="unstructured 100M clustered points, two cavities, 2,097,152 anisotropic Gaussians, forward"),
}


def mixture_for(w: Workload) -> Optional[Mixture]:
    """The point/mean density of a workload (built deterministically)."""
    if w.cfg == 2:
        m = _c3_mix()
    elif w.cfg == 3:
        m = _c4_mix()
    elif w.cfg == 4:
        m = _c5_mix()
    else:
        return None
    return m.build(rng(w.cfg, S_COMP))


def make_gaussians(w: Workload, n: Optional[int] = None) -> Gaussians:
    """Gaussian parameters of a workload: means (uniform or from the
    workload's density), per-axis log-normal scales, uniformly random unit
    quaternions (normalised standard normals), values U[0,1] and weights
    sigmoid(N(0,1))."""
    n = w.n_gauss if n is None else n
    g_mean = rng(w.cfg, S_MEAN)
    mean = g_mean.random((n, 3))
    if w.mean_mix_frac > 0.0:
        mix = mixture_for(w)
        g_mix = rng(w.cfg, S_MEANMIX)
        from_mix = g_mix.random(n) < w.mean_mix_frac
        k = int(from_mix.sum())
        mean[from_mix] = mix.sample(g_mix, k)
    log_s = rng(w.cfg, S_LOGSCALE).normal(w.log_scale_mu, w.log_scale_sd, size=(n, 3))
    q = rng(w.cfg, S_QUAT).standard_normal((n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    value = rng(w.cfg, S_VALUE).random(n)
    z = rng(w.cfg, S_WEIGHT).standard_normal(n)
    weight = 1.0 / (1.0 + np.exp(-z))
    f = np.float32
    return Gaussians(mean.astype(f), np.exp(log_s).astype(f), q.astype(f), value.astype(f), weight.astype(f))


def make_points(w: Workload, n: Optional[int] = None) -> np.ndarray:
    """Unstructured query cloud of a points workload, float32 [n,3]."""
    assert w.kind == "points"
    n = w.n_points if n is None else n
    mix = mixture_for(w)
    return mix.sample(rng(w.cfg, S_POINTS), n, dtype=np.float32)


def batch_permutation(w: Workload, total: int) -> np.ndarray:
    """Seeded permutation used to cut query batches (voxel ids or point ids)."""
    return rng(w.cfg, S_BATCH).permutation(total)


def voxel_batch(w: Workload) -> np.ndarray:
    """First `batch` entries of a seeded permutation of all voxel ids
    (x fastest), without replacement, left in random order; uint32."""
    total = w.dims[0] * w.dims[1] * w.dims[2]
    return batch_permutation(w, total)[: w.batch].astype(np.uint32)


def cotangents(w: Workload, n: int, batch_index: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """iid N(0,1) cotangents for the sampled value and the sampled influence."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(w.cfg, S_COTAN, batch_index))))
    gv = g.standard_normal(n).astype(np.float32)
    gi = g.standard_normal(n).astype(np.float32)
    return gv, gi


def jitter_offsets(cfg: int, n: int, iteration: int = 0) -> np.ndarray:
    """Training-sample offsets u in [0, 1)^3 per voxel (a random position in
    each voxel every iteration), drawn directly in float32 so that u < 1."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(cfg, S_JITTER, iteration))))
    return g.random((n, 3), dtype=np.float32)


def raw_params(w: Workload, n: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Free parameters behind make_gaussians, before the activations:
    log-scales [n,3] (the same draws), value logits log(v / (1 - v)) of the
    same U[0,1] values (clipped to [1e-6, 1 - 1e-6]) and weight logits (the
    same standard normals); float32."""
    n = w.n_gauss if n is None else n
    log_s = rng(w.cfg, S_LOGSCALE).normal(w.log_scale_mu, w.log_scale_sd, size=(n, 3))
    v = np.clip(rng(w.cfg, S_VALUE).random(n), 1e-6, 1.0 - 1e-6)
    z = rng(w.cfg, S_WEIGHT).standard_normal(n)
    f = np.float32
    return log_s.astype(f), np.log(v / (1.0 - v)).astype(f), z.astype(f)


def targets(cfg: int, n: int, iteration: int = 0) -> np.ndarray:
    """Target values of a training batch, U[0,1] float32 (the ground truth a
    structured volume would give at the samples)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(cfg, S_TARGET, iteration))))
    return g.random(n, dtype=np.float32)


def random_gaussians(seed: int, n: int, log_mu: float = np.log(0.05), log_sd: float = 0.3,
                     lo: float = 0.0, hi: float = 1.0) -> Gaussians:
    """Small free-form parameter sets for unit tests."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(1000, seed))))
    mean = g.uniform(lo, hi, size=(n, 3))
    s = np.exp(g.normal(log_mu, log_sd, size=(n, 3)))
    q = g.standard_normal((n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    v = g.random(n)
    w = 1.0 / (1.0 + np.exp(-g.standard_normal(n)))
    f = np.float32
    return Gaussians(mean.astype(f), s.astype(f), q.astype(f), v.astype(f), w.astype(f))


def random_points(seed: int, n: int, lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(2000, seed))))
    return g.uniform(lo, hi, size=(n, 3)).astype(np.float32)


def random_normal(seed: int, n: int) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=(3000, seed))))
    return g.standard_normal(n).astype(np.float32)
