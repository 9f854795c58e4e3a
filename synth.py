"""Seeded synthetic workloads for the permutohedral-lattice filter.

This module only draws input arrays (embeddings f, values v, upstream
gradients g).  It holds none of the filter's arithmetic, so both the GPU
path and the CPU oracle can be fed from it without sharing any code of the
method itself.

The paper trains on CT patches of 160x160x96 voxels (Section 3,
"Implementation details") whose embeddings come from a 1x1x1 convolution
over trunk features concatenated with a coordinate mesh (Fig. 2 caption).
The dataset and trained weights are not available, so each workload is a
synthetic volume of the same kind of shape: the embedding holds the voxel
coordinates divided by a spatial scale sigma_s, plus "learned-like" extra
channels:

* ``mix``: K blob centres drawn uniformly in the volume; each voxel takes
  the component of its nearest centre (ties to the lower index), whose mean
  is drawn from U[-3, 3]^m; the channel value is that mean plus i.i.d.
  N(0, std^2) noise.
* ``intensity``: i.i.d. N(0,1) noise, Gaussian-smoothed with sigma = 4
  voxels (reflecting boundary), standardised to zero mean and unit std and
  scaled by 3.

Values v and upstream gradients g are i.i.d. N(0, 1) in fp32.

Voxel order is x fastest: i = x + W*(y + H*z).
Seeds: 1907000 + 10*config + stream, stream 0 = embedding extras,
1 = values, 2 = upstream gradient; volume b of a batch adds 100*b.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 1907000


@dataclass(frozen=True)
class Workload:
    """One synthetic filtering problem (one or more independent volumes)."""

    name: str
    shape: tuple  # (W, H, D), x fastest
    sigma_s: float
    channels: int  # C, value channels
    extras: tuple = ()  # ("mix", m, K, std) or ("intensity", m)
    batch: int = 1
    backward: bool = True
    index: int = 0  # seed slot
    note: str = ""

    @property
    def d(self) -> int:
        m = 0
        for e in self.extras:
            m += e[1]
        return 3 + m

    @property
    def voxels(self) -> int:
        W, H, D = self.shape
        return W * H * D

    @property
    def total_voxels(self) -> int:
        return self.voxels * self.batch


WORKLOADS = {
    "C1": Workload("C1", (32, 32, 32), 4.0, 8, (), 1, False, 1,
                   "32^3, d=3 coordinates/4, C=8, forward only"),
    "C2": Workload("C2", (64, 64, 64), 8.0, 16, (("mix", 2, 6, 0.5),), 1, True, 2,
                   "64^3, d=5 = coordinates/8 + 2 mixture channels, C=16"),
    "C3": Workload("C3", (128, 128, 128), 16.0, 32, (("mix", 2, 6, 0.5),), 1, True, 3,
                   "128^3, d=5 = coordinates/16 + 2 mixture channels, C=32"),
    "C4": Workload("C4", (160, 160, 96), 16.0, 16, (("mix", 5, 10, 0.4),), 2, True, 4,
                   "2 x 160x160x96, d=8 = coordinates/16 + 5 mixture channels, C=16"),
    "C5": Workload("C5", (192, 192, 192), 24.0, 64, (("intensity", 1),), 1, True, 5,
                   "192^3, d=4 = coordinates/24 + 1 intensity channel, C=64"),
}


def seed(index: int, stream: int, volume: int = 0) -> int:
    return SEED_BASE + 10 * index + stream + 100 * volume


def coordinates(shape, sigma_s: float) -> np.ndarray:
    """N x 3 fp32 array of (x, y, z) / sigma_s with x fastest."""
    W, H, D = shape
    z, y, x = np.meshgrid(np.arange(D), np.arange(H), np.arange(W), indexing="ij")
    xyz = np.stack([x.ravel(), y.ravel(), z.ravel()], axis=1).astype(np.float64)
    return (xyz / sigma_s).astype(np.float32)


def mixture_channels(shape, m: int, K: int, std: float, rng) -> np.ndarray:
    W, H, D = shape
    centres = rng.uniform([0.0, 0.0, 0.0], [W, H, D], size=(K, 3))
    means = rng.uniform(-3.0, 3.0, size=(K, m))
    z, y, x = np.meshgrid(np.arange(D), np.arange(H), np.arange(W), indexing="ij")
    pos = np.stack([x.ravel(), y.ravel(), z.ravel()], axis=1).astype(np.float64)
    best = np.full(pos.shape[0], np.inf)
    comp = np.zeros(pos.shape[0], dtype=np.int64)
    for k in range(K):  # strict < keeps the lower index on ties
        dist = ((pos - centres[k]) ** 2).sum(axis=1)
        take = dist < best
        best[take] = dist[take]
        comp[take] = k
    noise = rng.standard_normal((pos.shape[0], m))
    return (means[comp] + std * noise).astype(np.float32)


def intensity_channel(shape, rng) -> np.ndarray:
    from scipy.ndimage import gaussian_filter

    W, H, D = shape
    vol = rng.standard_normal((D, H, W))
    vol = gaussian_filter(vol, sigma=4.0, mode="reflect")
    vol = (vol - vol.mean()) / vol.std()
    return (3.0 * vol).reshape(-1, 1).astype(np.float32)


def make_embedding(shape, sigma_s: float, extras=(), rng=None) -> np.ndarray:
    parts = [coordinates(shape, sigma_s)]
    for e in extras:
        if e[0] == "mix":
            parts.append(mixture_channels(shape, e[1], e[2], e[3], rng))
        elif e[0] == "intensity":
            parts.append(intensity_channel(shape, rng))
        else:
            raise ValueError(f"unknown extra channel kind {e[0]!r}")
    return np.ascontiguousarray(np.concatenate(parts, axis=1), dtype=np.float32)


def gaussian(n: int, c: int, s: int) -> np.ndarray:
    return np.random.default_rng(s).standard_normal((n, c), dtype=np.float32)


def generate(w: Workload | str, volume: int = 0, shape=None):
    """Return dict(f, v, g) for one volume of workload ``w``.

    ``shape`` overrides the volume shape (smaller test cases keep the same
    recipe and seeds)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    shp = tuple(shape) if shape is not None else w.shape
    rng = np.random.default_rng(seed(w.index, 0, volume))
    f = make_embedding(shp, w.sigma_s, w.extras, rng)
    n = f.shape[0]
    v = gaussian(n, w.channels, seed(w.index, 1, volume))
    g = gaussian(n, w.channels, seed(w.index, 2, volume))
    return {"f": f, "v": v, "g": g}


def random_points(n: int, d: int, scale: float, s: int) -> np.ndarray:
    """n x d fp32 points drawn uniformly in [0, scale)^d (small tests)."""
    rng = np.random.default_rng(s)
    return rng.uniform(0.0, scale, size=(n, d)).astype(np.float32)
