"""CPU oracle of the permutohedral block's prologue (Section 3 and the
Fig. 2 caption): the feature extractor is a 1x1x1 convolution of the
input channels with a mesh of spatial coordinates appended, followed by a
Leaky-ReLU; the descriptor extractor is a 1x1x1 convolution of the input
channels; features and descriptors are then split channel-wise into groups
and the module runs on each group independently.

TEST INFRASTRUCTURE ONLY: imported by the tests and the benchmark's CPU
baseline, never by the GPU library or its binding.  Plain numpy in fp64,
written from those definitions.

Layouts: x is N x c_in with voxel i = x + W (y + H z) (x fastest); the mesh
channels of voxel i are mesh_scale * (x, y, z); wf is d_tot x (c_in + 3)
(input columns: the c_in channels, then the mesh x, y, z), wv is
c_tot x c_in.  Outputs are in the grouped layout a batched lattice build
takes: group g holds rows [g N, (g+1) N) with channels
[g d_tot/G, (g+1) d_tot/G) of the features (likewise for the descriptors).
"""
from __future__ import annotations

import numpy as np


def mesh(dims, mesh_scale: float) -> np.ndarray:
    """N x 3 voxel coordinates (x, y, z) times mesh_scale, x fastest."""
    W, H, D = dims
    i = np.arange(W * H * D)
    return np.stack([i % W, (i // W) % H, i // (W * H)], axis=1).astype(np.float64) * mesh_scale


def to_groups(a: np.ndarray, groups: int) -> np.ndarray:
    """N x (G k) -> (G N) x k: group g's channels as rows g N .. (g+1) N - 1."""
    n, ch = a.shape
    k = ch // groups
    return np.concatenate([a[:, g * k:(g + 1) * k] for g in range(groups)], axis=0)


def from_groups(a: np.ndarray, groups: int) -> np.ndarray:
    """(G N) x k -> N x (G k), the inverse of to_groups."""
    n = a.shape[0] // groups
    return np.concatenate([a[g * n:(g + 1) * n] for g in range(groups)], axis=1)


def prologue_fwd(x, dims, wf, bf, wv, bv, mesh_scale: float, slope: float, groups: int):
    """Returns (features (G N) x d_tot/G, descriptors (G N) x c_tot/G)."""
    x = np.asarray(x, dtype=np.float64)
    xm = np.concatenate([x, mesh(dims, mesh_scale)], axis=1)
    z = xm @ np.asarray(wf, dtype=np.float64).T + np.asarray(bf, dtype=np.float64)
    f = np.where(z > 0, z, slope * z)
    v = x @ np.asarray(wv, dtype=np.float64).T + np.asarray(bv, dtype=np.float64)
    return to_groups(f, groups), to_groups(v, groups)


def prologue_bwd(x, dims, wf, bf, wv, mesh_scale: float, slope: float, groups: int, grad_f, grad_v):
    """Gradients of the prologue for upstream gradients in the grouped
    layout.  Returns (dx, dwf, dbf, dwv, dbv)."""
    x = np.asarray(x, dtype=np.float64)
    wf = np.asarray(wf, dtype=np.float64)
    wv = np.asarray(wv, dtype=np.float64)
    xm = np.concatenate([x, mesh(dims, mesh_scale)], axis=1)
    z = xm @ wf.T + np.asarray(bf, dtype=np.float64)
    dz = from_groups(np.asarray(grad_f, dtype=np.float64), groups) * np.where(z > 0, 1.0, slope)
    dv = from_groups(np.asarray(grad_v, dtype=np.float64), groups)
    c_in = x.shape[1]
    dx = dz @ wf[:, :c_in] + dv @ wv
    return dx, dz.T @ xm, dz.sum(axis=0), dv.T @ x, dv.sum(axis=0)
