"""Pins of the permutohedral-block prologue oracle (Section 3, Fig. 2
caption: 1x1x1 feature convolution over the input channels plus a mesh of
spatial coordinates, Leaky-ReLU; 1x1x1 descriptor convolution; channel
groups)."""
import numpy as np
import pytest

import synth
from oracle import block as B


def case(dims=(5, 4, 3), c_in=6, d_tot=4, c_tot=6, groups=2, seed=0):
    rng = np.random.default_rng(seed)
    n = dims[0] * dims[1] * dims[2]
    x = rng.standard_normal((n, c_in))
    wf = rng.standard_normal((d_tot, c_in + 3)) * 0.5
    bf = rng.standard_normal(d_tot) * 0.3
    wv = rng.standard_normal((c_tot, c_in)) * 0.5
    bv = rng.standard_normal(c_tot) * 0.3
    return x, wf, bf, wv, bv


def test_mesh_is_the_workload_coordinate_recipe():
    """With the feature convolution selecting the mesh channels, zero
    input weights and a bias keeping the Leaky-ReLU on its linear side, the
    features are the voxel coordinates / sigma_s of the synthetic volumes."""
    dims, sig = (7, 5, 4), 8.0
    n = 7 * 5 * 4
    x = np.random.default_rng(1).standard_normal((n, 2))
    wf = np.zeros((3, 5))
    wf[:, 2:] = np.eye(3)
    f, _ = B.prologue_fwd(x, dims, wf, np.zeros(3), np.zeros((2, 2)), np.zeros(2), 1.0 / sig, 0.01, 1)
    np.testing.assert_allclose(f, synth.coordinates(dims, sig).astype(np.float64), rtol=1e-6, atol=1e-7)
    # the negative side: -coordinates come out scaled by the slope
    f2, _ = B.prologue_fwd(x, dims, -wf, np.full(3, -1e-3), np.zeros((2, 2)), np.zeros(2), 1.0 / sig, 0.2, 1)
    np.testing.assert_allclose(f2, 0.2 * (-synth.coordinates(dims, sig).astype(np.float64) - 1e-3), rtol=1e-6,
                               atol=1e-7)


def test_groups_layout():
    """Group g holds rows [g N, (g+1) N) with its slice of the channels."""
    x, wf, bf, wv, bv = case(groups=2)
    f, v = B.prologue_fwd(x, (5, 4, 3), wf, bf, wv, bv, 0.25, 0.01, 2)
    f1, v1 = B.prologue_fwd(x, (5, 4, 3), wf, bf, wv, bv, 0.25, 0.01, 1)
    n = 60
    np.testing.assert_array_equal(f[:n], f1[:, :2])
    np.testing.assert_array_equal(f[n:], f1[:, 2:])
    np.testing.assert_array_equal(v[n:], v1[:, 3:])
    np.testing.assert_array_equal(B.from_groups(f, 2), f1)


@pytest.mark.parametrize("groups", [1, 2])
def test_prologue_gradients_finite_differences(groups):
    """Central differences of L = <gf, f> + <gv, v> in every parameter and
    a sample of inputs (the Leaky-ReLU is linear away from its kink; points
    within 1e-3 of it are avoided)."""
    dims = (4, 3, 3)
    x, wf, bf, wv, bv = case(dims=dims, groups=groups, seed=3)
    rng = np.random.default_rng(4)
    f0, v0 = B.prologue_fwd(x, dims, wf, bf, wv, bv, 0.3, 0.05, groups)
    gf = rng.standard_normal(f0.shape)
    gv = rng.standard_normal(v0.shape)

    def L(x_, wf_, bf_, wv_, bv_):
        f, v = B.prologue_fwd(x_, dims, wf_, bf_, wv_, bv_, 0.3, 0.05, groups)
        return float((gf * f).sum() + (gv * v).sum())

    dx, dwf, dbf, dwv, dbv = B.prologue_bwd(x, dims, wf, bf, wv, 0.3, 0.05, groups, gf, gv)
    xm = np.concatenate([x, B.mesh(dims, 0.3)], axis=1)
    assert np.abs(xm @ wf.T + bf).min() > 1e-3
    h = 1e-6
    args = [x, wf, bf, wv, bv]
    grads = [dx, dwf, dbf, dwv, dbv]
    for a, (arr, gr) in enumerate(zip(args, grads)):
        flat = arr.reshape(-1)
        for idx in range(0, flat.size, max(1, flat.size // 25)):
            old = flat[idx]
            flat[idx] = old + h
            lp = L(*args)
            flat[idx] = old - h
            lm = L(*args)
            flat[idx] = old
            assert (lp - lm) / (2 * h) == pytest.approx(gr.reshape(-1)[idx], rel=1e-6, abs=1e-7), (a, idx)


def test_planted_wrong_slope_side_breaks_finite_differences():
    """Using the slope on the positive side of the Leaky-ReLU fails the
    finite-difference pin."""
    dims = (4, 3, 2)
    x, wf, bf, wv, bv = case(dims=dims, groups=1, seed=5)
    gf = np.random.default_rng(6).standard_normal((24, 4))
    gv = np.zeros((24, 6))
    xm = np.concatenate([x, B.mesh(dims, 0.3)], axis=1)
    z = xm @ wf.T + bf
    dz_wrong = gf * np.where(z > 0, 0.05, 1.0)
    _, dwf, _, _, _ = B.prologue_bwd(x, dims, wf, bf, wv, 0.3, 0.05, 1, gf, gv)
    assert np.abs(dz_wrong.T @ xm - dwf).max() > 1e-3
