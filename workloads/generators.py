"""Seeded synthetic point-cloud workloads.

This module only synthesises inputs. It holds none of the loss's arithmetic and
is shared by the tests, the benchmark and the smoke check, so that the CPU
reference and the GPU library always see bit-identical float32 inputs.

The paper evaluates on ShapeNet-34/55, PCN and MM-Fi (Sec. IV-A). None of those
datasets is used here: the generators below produce stand-ins with the same
shapes and a similar geometric structure (object surfaces, partial/noisy
predictions, unequal cardinalities, scene-scale clusters).

Every sample b of configuration `cfg` is drawn from
``numpy.random.default_rng(SeedSequence([20251219, cfg, b]))`` in float64 and
rounded once to float32.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, Optional, Sequence, Tuple

import numpy as np

SEED = 20251219


@dataclasses.dataclass(frozen=True)
class Workload:
    """One benchmark configuration: batch shape, Sinkhorn length and recipe."""

    cfg: int
    name: str
    B: int
    N: int
    M: int
    n_iter: int
    reference: str  # 'sphere' | 'primitives' | 'gmm'
    prediction: str  # 'perm_noise' | 'uniform_cube'
    sigma: float

    @property
    def pairs(self) -> int:
        return self.B * self.N * self.M


CONFIGS: Dict[int, Workload] = {
    1: Workload(1, "tiny", 2, 256, 256, 10, "sphere", "perm_noise", 0.02),
    2: Workload(2, "shape-completion", 32, 2048, 2048, 10, "primitives", "perm_noise", 0.05),
    3: Workload(3, "large-batch", 64, 8192, 8192, 20, "primitives", "perm_noise", 0.01),
    4: Workload(4, "unequal", 16, 4096, 16384, 10, "primitives", "uniform_cube", 0.0),
    5: Workload(5, "large-scene", 4, 65536, 65536, 10, "gmm", "perm_noise", 0.05),
}


def rng_for(cfg: int, b: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED, int(cfg), int(b)]))


# --------------------------------------------------------------------------
# surfaces
# --------------------------------------------------------------------------

def random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Uniformly distributed rotation matrix from a normalised 4-D Gaussian quaternion."""
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array(
        [
            [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
            [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
            [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
        ]
    )


def sphere_surface(rng: np.random.Generator, n: int, radius: float = 1.0) -> np.ndarray:
    v = rng.standard_normal((n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    return v * radius


def _box_surface(rng, n, h):
    # six faces, two per axis; pick a face with probability proportional to its area
    areas = np.array([h[1] * h[2], h[1] * h[2], h[0] * h[2], h[0] * h[2], h[0] * h[1], h[0] * h[1]])
    face = rng.choice(6, size=n, p=areas / areas.sum())
    u = rng.uniform(-1.0, 1.0, size=(n, 3)) * h
    axis = face // 2
    sign = np.where(face % 2 == 0, 1.0, -1.0)
    u[np.arange(n), axis] = sign * h[axis]
    return u


def _cylinder_surface(rng, n, r, hh):
    side, cap = 2 * np.pi * r * 2 * hh, np.pi * r * r
    part = rng.choice(3, size=n, p=np.array([side, cap, cap]) / (side + 2 * cap))
    out = np.empty((n, 3))
    theta = rng.uniform(0, 2 * np.pi, size=n)
    rad = np.where(part == 0, r, r * np.sqrt(rng.uniform(0, 1, size=n)))
    out[:, 0] = rad * np.cos(theta)
    out[:, 1] = rad * np.sin(theta)
    out[:, 2] = np.where(part == 0, rng.uniform(-hh, hh, size=n), np.where(part == 1, hh, -hh))
    return out


def primitive_surface(rng: np.random.Generator, n: int) -> np.ndarray:
    """Surface samples of a random union of 1-4 spheres/boxes/cylinders in the unit ball."""
    k = int(rng.integers(1, 5))
    kinds = rng.integers(0, 3, size=k)
    params, areas = [], []
    for kind in kinds:
        if kind == 0:
            r = rng.uniform(0.2, 0.6)
            params.append(("sphere", r))
            areas.append(4 * np.pi * r * r)
        elif kind == 1:
            h = rng.uniform(0.1, 0.6, size=3)
            params.append(("box", h))
            areas.append(8 * (h[0] * h[1] + h[1] * h[2] + h[0] * h[2]))
        else:
            r, hh = rng.uniform(0.1, 0.5), rng.uniform(0.1, 0.6)
            params.append(("cylinder", (r, hh)))
            areas.append(2 * np.pi * r * 2 * hh + 2 * np.pi * r * r)
    areas = np.asarray(areas)
    counts = rng.multinomial(n, areas / areas.sum())
    parts = []
    for (kind, prm), c in zip(params, counts):
        if c == 0:
            continue
        if kind == "sphere":
            p = sphere_surface(rng, c, prm)
        elif kind == "box":
            p = _box_surface(rng, c, prm)
        else:
            p = _cylinder_surface(rng, c, *prm)
        p = p @ random_rotation(rng).T + rng.uniform(-0.5, 0.5, size=3)
        parts.append(p)
    pts = np.concatenate(parts, axis=0)
    pts = pts - pts.mean(axis=0)
    pts /= np.linalg.norm(pts, axis=1).max()
    return pts


def gmm_scene(rng: np.random.Generator, n: int, clusters: int = 64) -> np.ndarray:
    """Anisotropic Gaussian mixture: means in [-10,10]^3, covariance eigenvalues in [0.01,1]."""
    means = rng.uniform(-10, 10, size=(clusters, 3))
    chol = []
    for _ in range(clusters):
        R = random_rotation(rng)
        lam = rng.uniform(0.01, 1.0, size=3)
        chol.append(R * np.sqrt(lam))  # R diag(sqrt(lam)): cov = R diag(lam) R^T
    label = rng.integers(0, clusters, size=n)
    z = rng.standard_normal((n, 3))
    out = np.empty((n, 3))
    for c in range(clusters):
        m = label == c
        out[m] = z[m] @ chol[c].T + means[c]
    return out


def _reference(rng, kind: str, m: int) -> np.ndarray:
    if kind == "sphere":
        return sphere_surface(rng, m)
    if kind == "primitives":
        return primitive_surface(rng, m)
    if kind == "gmm":
        return gmm_scene(rng, m)
    raise ValueError(kind)


def _prediction(rng, kind: str, ref: np.ndarray, n: int, sigma: float) -> np.ndarray:
    if kind == "perm_noise":
        assert n == ref.shape[0], "a permuted prediction needs N == M"
        return ref[rng.permutation(n)] + rng.normal(0.0, sigma, size=(n, 3))
    if kind == "uniform_cube":
        return rng.uniform(-1.0, 1.0, size=(n, 3))
    raise ValueError(kind)


def sample(w: Workload, b: int) -> Tuple[np.ndarray, np.ndarray]:
    """Sample b of workload w as float32 (N,3) prediction and (M,3) reference."""
    rng = rng_for(w.cfg, b)
    y = _reference(rng, w.reference, w.M)
    x = _prediction(rng, w.prediction, y, w.N, w.sigma)
    return np.ascontiguousarray(x, dtype=np.float32), np.ascontiguousarray(y, dtype=np.float32)


def batch(w: Workload, samples: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Float32 arrays X (B,N,3) and Y (B,M,3) for the listed samples (default: all B)."""
    idx = range(w.B) if samples is None else samples
    xs, ys = zip(*(sample(w, b) for b in idx))
    return np.stack(xs), np.stack(ys)


def config(cfg: int, **overrides) -> Workload:
    """Configuration `cfg`, optionally with some fields replaced (e.g. a smaller B)."""
    return dataclasses.replace(CONFIGS[cfg], **overrides)


def custom(seed: int, B: int, N: int, M: int, reference: str = "sphere",
           prediction: str = "perm_noise", sigma: float = 0.02) -> Tuple[np.ndarray, np.ndarray]:
    """Ad-hoc seeded case for edge/ragged tests; N != M requires prediction='uniform_cube'
    or a reference of size N (the permuted prediction then uses the first N reference points)."""
    xs, ys = [], []
    for b in range(B):
        rng = np.random.default_rng(np.random.SeedSequence([SEED, 1000 + seed, B, N, M, b]))
        y = _reference(rng, reference, M)
        if prediction == "perm_noise" and N != M:
            base = y[rng.permutation(M)[:N]] if N <= M else y[rng.integers(0, M, size=N)]
            x = base + rng.normal(0.0, sigma, size=(N, 3))
        else:
            x = _prediction(rng, prediction, y, N, sigma)
        xs.append(x.astype(np.float32))
        ys.append(y.astype(np.float32))
    return np.ascontiguousarray(np.stack(xs)), np.ascontiguousarray(np.stack(ys))
