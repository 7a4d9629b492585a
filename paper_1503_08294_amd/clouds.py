"""Seeded synthetic point clouds, initial units and signal streams.

The paper reconstructs surfaces from point clouds sampled uniformly from triangular meshes
(Sec. 3.1); those meshes are not available, so these generators stand in for them with
analytic surfaces of comparable genus and density structure.  This module holds no step of
the method: it only produces inputs, which both the HIP path and the CPU oracle consume.
Everything is drawn with ``numpy.random.default_rng`` in float64 and cast to float32 at the
end.  Signals are drawn i.i.d. with replacement from the cloud (Sec. 2.1 "Sample").
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

TWO_PI = 2.0 * np.pi


# ----------------------------------------------------------------------- surfaces ----

def sphere_cloud(n_points: int, seed: int, radius: float = 1.0,
                 center=(0.0, 0.0, 0.0)) -> np.ndarray:
    """Uniform on a sphere: normalised standard-normal vectors.  Returns (n, 3) float32."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((n_points, 3))
    g /= np.linalg.norm(g, axis=1, keepdims=True)
    return (np.asarray(center) + radius * g).astype(np.float32)


def _torus_points(rng, n: int, R: float, r: float) -> np.ndarray:
    """Area-uniform on a torus: theta uniform, phi by rejection with acceptance
    (R + r cos phi) / (R + r), which is proportional to the area element."""
    out = np.empty((0, 3))
    while out.shape[0] < n:
        k = max(16, int((n - out.shape[0]) * 1.6))
        phi = rng.uniform(0.0, TWO_PI, k)
        keep = rng.uniform(0.0, 1.0, k) < (R + r * np.cos(phi)) / (R + r)
        phi = phi[keep]
        theta = rng.uniform(0.0, TWO_PI, phi.shape[0])
        rho = R + r * np.cos(phi)
        p = np.stack([rho * np.cos(theta), rho * np.sin(theta), r * np.sin(phi)], axis=1)
        out = np.concatenate([out, p])
    return out[:n]


def torus_cloud(n_points: int, seed: int, R: float = 1.0, r: float = 0.3,
                sigma: float = 0.005) -> np.ndarray:
    """Torus (R, r) sampled area-uniformly plus isotropic Gaussian noise."""
    rng = np.random.default_rng(seed)
    p = _torus_points(rng, n_points, R, r)
    if sigma > 0:
        p = p + rng.normal(0.0, sigma, p.shape)
    return p.astype(np.float32)


_BALLS = (((-0.45, 0.0, 0.0), 0.6), ((0.45, 0.0, 0.0), 0.6), ((0.0, 0.55, 0.0), 0.5))
_BALL_WEIGHTS = (10.0, 1.0, 3.0)
_PATCH = (-0.8, 1.2, 1.0)  # plane z = -0.8, |x|, |y| <= 1.2, weight 1


def spheres_plane_cloud(n_points: int, seed: int) -> np.ndarray:
    """Boundary of a union of three pairwise-intersecting balls plus a square plane patch
    below them.  Regions are chosen with probability proportional to weight x area (weights
    10 : 1 : 3 on the spheres, 1 on the patch, so densities differ 10 : 1); points on a
    sphere that fall strictly inside another ball are rejected."""
    rng = np.random.default_rng(seed)
    areas = [4.0 * np.pi * r * r for _, r in _BALLS]
    z0, half, w_patch = _PATCH
    areas.append((2.0 * half) ** 2)
    weights = np.array(list(_BALL_WEIGHTS) + [w_patch]) * np.array(areas)
    prob = weights / weights.sum()
    out = np.empty((0, 3))
    while out.shape[0] < n_points:
        k = max(64, int((n_points - out.shape[0]) * 1.3))
        region = rng.choice(4, size=k, p=prob)
        pts = np.empty((k, 3))
        for i, (c, r) in enumerate(_BALLS):
            sel = region == i
            g = rng.standard_normal((int(sel.sum()), 3))
            g /= np.linalg.norm(g, axis=1, keepdims=True)
            pts[sel] = np.asarray(c) + r * g
        sel = region == 3
        cnt = int(sel.sum())
        pts[sel] = np.stack([rng.uniform(-half, half, cnt), rng.uniform(-half, half, cnt),
                             np.full(cnt, z0)], axis=1)
        keep = np.ones(k, bool)
        for i, (c, r) in enumerate(_BALLS):
            inside = np.linalg.norm(pts - np.asarray(c), axis=1) < r - 1e-9
            keep &= ~(inside & (region != i))
        out = np.concatenate([out, pts[keep]])
    return out[:n_points].astype(np.float32)


# Genus-3 tube surface: points at distance TUBE from the graph G made of the unit circle
# in z = 0 and the two chords x = +-CHORD_X.  G has 4 vertices and 6 edges, so its cycle
# rank, and the genus of the tube surface around it, is 3.
GENUS3_TUBE = 0.12
GENUS3_CHORD_X = 0.35


def _dist_to_circle(p: np.ndarray) -> np.ndarray:
    rho = np.hypot(p[:, 0], p[:, 1])
    return np.hypot(rho - 1.0, p[:, 2])


def _dist_to_chord(p: np.ndarray, x0: float) -> np.ndarray:
    h = np.sqrt(1.0 - x0 * x0)
    yc = np.clip(p[:, 1], -h, h)
    return np.sqrt((p[:, 0] - x0) ** 2 + (p[:, 1] - yc) ** 2 + p[:, 2] ** 2)


def genus3_distance(p: np.ndarray) -> np.ndarray:
    """Distance from each point to the skeleton graph G (float64)."""
    p = np.asarray(p, np.float64)
    return np.minimum(_dist_to_circle(p),
                      np.minimum(_dist_to_chord(p, GENUS3_CHORD_X),
                                 _dist_to_chord(p, -GENUS3_CHORD_X)))


def genus3_cloud(n_points: int, seed: int, jitter: float = 0.002) -> np.ndarray:
    """Area-uniform samples of the zero set of F(p) = dist(p, G) - TUBE, plus jitter.
    Each primitive's tube (a torus for the circle, open cylinders for the chords) is
    sampled area-uniformly with probability proportional to its area, and points closer
    than TUBE to G (inside another primitive's tube) are rejected."""
    rng = np.random.default_rng(seed)
    r = GENUS3_TUBE
    h = np.sqrt(1.0 - GENUS3_CHORD_X ** 2)
    a_torus = 4.0 * np.pi ** 2 * 1.0 * r
    a_cyl = TWO_PI * r * 2.0 * h
    prob = np.array([a_torus, a_cyl, a_cyl])
    prob /= prob.sum()
    out = np.empty((0, 3))
    while out.shape[0] < n_points:
        k = max(64, int((n_points - out.shape[0]) * 1.4))
        which = rng.choice(3, size=k, p=prob)
        pts = np.empty((k, 3))
        nt = int((which == 0).sum())
        pts[which == 0] = _torus_points(rng, nt, 1.0, r)
        for i, x0 in ((1, GENUS3_CHORD_X), (2, -GENUS3_CHORD_X)):
            sel = which == i
            c = int(sel.sum())
            t = rng.uniform(-h, h, c)
            a = rng.uniform(0.0, TWO_PI, c)
            pts[sel] = np.stack([x0 + r * np.cos(a), t, r * np.sin(a)], axis=1)
        keep = genus3_distance(pts) >= r - 1e-6
        out = np.concatenate([out, pts[keep]])
    out = out[:n_points]
    if jitter > 0:
        out = out + rng.normal(0.0, jitter, out.shape)
    return out.astype(np.float32)


# ----------------------------------------------------------------- units, signals ----

def initial_units(cloud: np.ndarray, n_units: int, seed: int) -> np.ndarray:
    """n distinct cloud points (without replacement), SoA (3, n) float32."""
    rng = np.random.default_rng(seed)
    idx = rng.choice(cloud.shape[0], size=n_units, replace=False)
    return np.ascontiguousarray(cloud[idx].T.astype(np.float32))


class SignalStream:
    """i.i.d. draws with replacement from the cloud, one batch of m per iteration, from a
    single Generator advanced across iterations.  Each batch is SoA (3, m) float32."""

    def __init__(self, cloud: np.ndarray, seed: int):
        self.cloud = np.asarray(cloud, np.float32)
        self.rng = np.random.default_rng(seed)

    def next(self, m: int) -> np.ndarray:
        idx = self.rng.integers(0, self.cloud.shape[0], m)
        return np.ascontiguousarray(self.cloud[idx].T)


# ------------------------------------------------------------------- workloads ----

@dataclass
class Workload:
    """One synthetic workload: cloud, initial units, run length and parameters."""
    name: str
    cloud: str
    n_points: int
    n_units: int
    m: int
    iterations: int
    max_age: int = 50
    insert_every: int = 0
    n_max: int = 0
    eps_b: float = 0.05
    eps_n: float = 0.0006
    err_alpha: float = 0.5
    err_beta: float = 0.995
    grow: bool = False
    sweep_m: tuple = field(default_factory=tuple)
    cloud_seed: int = 0
    unit_seed: int = 1
    signal_seed: int = 2

    def make_cloud(self, n_points: int | None = None) -> np.ndarray:
        n = self.n_points if n_points is None else n_points
        if self.cloud == "sphere":
            return sphere_cloud(n, self.cloud_seed)
        if self.cloud == "torus":
            return torus_cloud(n, self.cloud_seed, 1.0, 0.3, 0.005)
        if self.cloud == "spheres_plane":
            return spheres_plane_cloud(n, self.cloud_seed)
        if self.cloud == "genus3":
            return genus3_cloud(n, self.cloud_seed, 0.002)
        raise ValueError(self.cloud)

    def make_units(self, cloud: np.ndarray, n_units: int | None = None) -> np.ndarray:
        n = self.n_units if n_units is None else n_units
        if self.cloud == "sphere":
            # units at their own seeded points on the sphere, independent of the cloud
            return np.ascontiguousarray(sphere_cloud(n, self.unit_seed).T)
        return initial_units(cloud, n, self.unit_seed)

    def capacity(self, m_max: int | None = None) -> dict:
        n_max = max(self.n_max, self.n_units)
        return {"n_max": n_max, "e_max": 4 * n_max + 16,
                "m_max": m_max if m_max is not None else max((self.m,) + tuple(self.sweep_m))}


WORKLOADS = {
    "tiny_sphere": Workload("tiny_sphere", "sphere", 20_000, 1_000, 256, 20),
    "torus_grow": Workload("torus_grow", "torus", 200_000, 10_000, 2_048, 100,
                           insert_every=10, n_max=12_000, grow=True),
    "spheres_plane_prune": Workload("spheres_plane_prune", "spheres_plane", 1_000_000,
                                    50_000, 8_192, 200, max_age=8, insert_every=10,
                                    n_max=60_000, grow=True),
    "genus3_200k": Workload("genus3_200k", "genus3", 4_000_000, 200_000, 16_384, 100),
    "torus_sweep": Workload("torus_sweep", "torus", 2_000_000, 100_000, 16_384, 60,
                            sweep_m=(1, 64, 1_024, 16_384, 65_536)),
}
