"""Pins of the CPU oracle against facts that do not come from the oracle.

Every test here checks the oracle against mathematics the paper's method
fixes: closed forms, invariants of the lattice, a brute-force nearest point,
an independent 1-D textbook filter, the exact Gaussian sum it approximates,
the adjoint identity behind eq. (7) and finite differences for eq. (8).
The last block plants plausible mistakes in the oracle's composition and
shows that the pins catch them.
"""
import itertools
import math

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

DIMS = [1, 2, 3, 4, 5, 8]


def rel(a, b):
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300))


def full_keys(keys):
    """Append the implicit last coordinate (minus the sum of the stored ones)."""
    return np.concatenate([keys, -keys.sum(axis=-1, keepdims=True)], axis=-1)


def u_vec(d, j):
    u = -np.ones(d + 1, dtype=np.int64)
    u[j] = d
    return u


# --------------------------------------------------------------------------
# Embedding matrix (the position embedding matrix E of eq. 8)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", list(range(1, 17)))
def test_embedding_matrix_closed_form(O, d):
    E = O.embedding_matrix(d)
    a = O.alpha(d)
    assert a == pytest.approx((d + 1) * math.sqrt(2.0 / 3.0), rel=1e-15)
    np.testing.assert_allclose(E.T @ E, a * a * np.eye(d), atol=1e-12 * a * a)
    np.testing.assert_allclose(E.sum(axis=0), 0.0, atol=1e-12 * a)
    p = np.random.default_rng(d).standard_normal(d)
    assert np.linalg.norm(E @ p) == pytest.approx(a * np.linalg.norm(p), rel=1e-12)


# --------------------------------------------------------------------------
# Enclosing simplex
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", DIMS)
def test_simplex_invariants(O, d):
    f = synth.random_points(3000, d, 12.0, 100 + d) - 6.0
    s = O.simplex(f)
    K = full_keys(s.keys.astype(np.int64))           # n x (d+1) x (d+1)
    n = f.shape[0]
    # vertex k has every coordinate congruent to k mod d+1 and lies on sum(x)=0
    for k in range(d + 1):
        assert np.all(np.mod(K[:, k, :] - k, d + 1) == 0)
    # ranks are a permutation of 0..d
    assert np.all(np.sort(s.rank, axis=1) == np.arange(d + 1))
    # barycentric weights: nonnegative, sum to one, reproduce the point
    assert s.bary.min() > -1e-6
    np.testing.assert_allclose(s.bary.sum(axis=1), 1.0, atol=1e-12)
    recon = np.einsum("nk,nkc->nc", s.bary, K.astype(np.float64))
    scale = 1.0 + np.abs(s.xelev).max()
    np.testing.assert_allclose(recon, s.xelev, atol=1e-12 * scale)
    np.testing.assert_allclose(s.xelev, f.astype(np.float64) @ O.embedding_matrix(d).T,
                               atol=1e-12 * scale)
    # consecutive vertices differ by -u_c where c has rank d-k; the d+1 steps
    # form a cycle that uses every direction once
    for i in range(0, n, 97):
        for k in range(d + 1):
            c = int(np.where(s.rank[i] == d - k)[0][0])
            nxt = K[i, (k + 1) % (d + 1)] if k < d else K[i, 0]
            if k < d:
                assert np.array_equal(nxt - K[i, k], -u_vec(d, c))
            else:
                c0 = int(np.where(s.rank[i] == 0)[0][0])
                assert np.array_equal(K[i, 0] - K[i, d], -u_vec(d, c0))


@pytest.mark.parametrize("d", [1, 2, 3, 4, 5])
def test_remainder0_point_is_nearest(O, d):
    """Vertex 0 is the remainder-0 point; no other point of (d+1)A_d within
    one step on every coordinate is closer to the elevated position."""
    f = synth.random_points(400, d, 10.0, 200 + d) - 5.0
    s = O.simplex(f)
    K = full_keys(s.keys.astype(np.int64))
    r = K[:, 0, :]
    assert np.all(np.mod(r, d + 1) == 0) and np.all(r.sum(axis=1) == 0)
    zs = [np.array(z) for z in itertools.product((-1, 0, 1), repeat=d + 1) if sum(z) == 0]
    x = s.xelev
    best = ((x - r) ** 2).sum(axis=1)
    for z in zs:
        alt = ((x - (r + (d + 1) * z)) ** 2).sum(axis=1)
        assert np.all(best <= alt + 1e-9)


# --------------------------------------------------------------------------
# Sparse lattice: vertex set and neighbours by definition
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", [2, 3, 5, 8])
def test_dedup_and_neighbours_by_definition(O, d):
    f = synth.random_points(1500, d, 6.0, 300 + d)
    lat = O.lattice(f)
    allkeys = {tuple(k) for k in lat.simp.keys.reshape(-1, d).tolist()}
    assert lat.M == len(allkeys)
    assert [tuple(k) for k in lat.keys.tolist()] == sorted(allkeys)
    ids = {k: i for i, k in enumerate(sorted(allkeys))}
    # every (point, vertex) id points at its own key
    got = lat.keys[lat.vert.reshape(-1)]
    assert np.array_equal(got, lat.simp.keys.reshape(-1, d))
    for m in range(0, lat.M, max(1, lat.M // 300)):
        key = lat.keys[m].astype(np.int64)
        for j in range(d + 1):
            u = u_vec(d, j)[:d]
            assert lat.nbr[m, j, 0] == ids.get(tuple((key - u).tolist()), -1)
            assert lat.nbr[m, j, 1] == ids.get(tuple((key + u).tolist()), -1)
    # symmetric links: m's + neighbour along j has m as its - neighbour
    for m in range(lat.M):
        for j in range(d + 1):
            hi = lat.nbr[m, j, 1]
            if hi >= 0:
                assert lat.nbr[hi, j, 0] == m


# --------------------------------------------------------------------------
# Special case that reduces to a textbook filter: d = 1
# --------------------------------------------------------------------------

def textbook_1d(p, v, normalize):
    """Uniform 1-D grid with spacing sqrt(3)/2, tent splat, two [1 2 1]
    passes over the touched nodes (untouched nodes read as 0), tent slice.
    Raw mode divides by the kernel mass 16 * spacing / sqrt(2 pi)."""
    h = math.sqrt(3.0) / 2.0
    t = p / h
    lo = np.floor(t).astype(np.int64)
    fr = t - lo
    C = v.shape[1]
    L = {}
    for i in range(len(p)):
        for node, w in ((lo[i], 1.0 - fr[i]), (lo[i] + 1, fr[i])):
            L.setdefault(int(node), np.zeros(C))
            L[int(node)] = L[int(node)] + w * v[i]
    for _ in range(2):
        L = {a: L.get(a - 1, 0.0) + 2.0 * L[a] + L.get(a + 1, 0.0) for a in L}
    out = np.array([(1.0 - fr[i]) * L[int(lo[i])] + fr[i] * L[int(lo[i]) + 1] for i in range(len(p))])
    if normalize:
        return out
    return out / (16.0 * h / math.sqrt(2.0 * math.pi))


@pytest.mark.parametrize("normalize", [False, True])
def test_d1_matches_textbook_grid_filter(O, normalize):
    rng = np.random.default_rng(11)
    # clustered points with gaps, so that some grid nodes are absent
    p = np.concatenate([rng.uniform(0, 3, 40), rng.uniform(7, 8, 20), rng.uniform(20, 20.4, 5)])
    p = p.astype(np.float32)
    t = p.astype(np.float64) / (math.sqrt(3) / 2)
    keep = np.abs(t - np.round(t)) > 1e-4  # keep away from exact grid nodes
    p = p[keep]
    v = rng.standard_normal((len(p), 3))
    lat = O.lattice(p.reshape(-1, 1))
    out, _ = O.forward(lat, v, normalize)
    if normalize:
        ref = textbook_1d(p.astype(np.float64), v, True) / textbook_1d(p.astype(np.float64), np.ones((len(p), 1)), True)
    else:
        ref = textbook_1d(p.astype(np.float64), v, False)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# Closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", [1, 2, 3, 5, 8])
def test_single_point_closed_form(O, d):
    """One point: M = d+1 vertices in a cycle; each direction joins exactly
    one pair; raw out = s_d * b^T (prod_j (2I + N_j)) b * v with N_j built
    here from the keys alone."""
    p = (synth.random_points(1, d, 3.0, 400 + d) + 0.123).astype(np.float32)
    lat = O.lattice(p)
    assert lat.M == d + 1
    assert int((lat.nbr >= 0).sum()) == 2 * (d + 1)
    b = lat.simp.bary[0]
    K = full_keys(lat.simp.keys[0].astype(np.int64))
    B = np.eye(d + 1)
    for j in range(d + 1):
        Nj = np.zeros((d + 1, d + 1))
        u = u_vec(d, j)
        for a in range(d + 1):
            for c in range(d + 1):
                diff = K[c] - K[a]
                if np.array_equal(diff, u) or np.array_equal(diff, -u):
                    Nj[a, c] = 1.0
        assert Nj.sum() == 2.0
        B = (2.0 * np.eye(d + 1) + Nj) @ B
    gain = b @ B @ b
    v = np.array([[1.5, -2.0, 0.25]])
    out, _ = O.forward(lat, v, False)
    np.testing.assert_allclose(out, O.raw_scale(d) * gain * v, rtol=1e-13)
    outn, _ = O.forward(lat, v, True)
    np.testing.assert_allclose(outn, v, rtol=1e-13)


@pytest.mark.parametrize("d", [1, 2, 3, 4, 5, 8])
def test_raw_scale_closed_form(O, d):
    covol = 1.5 ** (d / 2.0) / math.sqrt(d + 1)  # lattice covolume in input units
    G = 4.0 ** (d + 1) * covol / (2 * math.pi) ** (d / 2.0)
    assert 1.0 / O.raw_scale(d) == pytest.approx(G, rel=1e-13)


@pytest.mark.parametrize("d", [2, 3, 5])
def test_far_apart_points_do_not_interact(O, d):
    rng = np.random.default_rng(500 + d)
    n = 12
    f = rng.uniform(0, 1, size=(n, d))
    f[:, 0] += 25.0 * np.arange(n)
    f = f.astype(np.float32)
    v = rng.standard_normal((n, 4))
    g = rng.standard_normal((n, 4))
    lat = O.lattice(f)
    out, st = O.forward(lat, v, False)
    dv, df = O.backward(lat, v, g, False, st)
    for i in range(n):
        li = O.lattice(f[i:i + 1])
        oi, si = O.forward(li, v[i:i + 1], False)
        dvi, dfi = O.backward(li, v[i:i + 1], g[i:i + 1], False, si)
        np.testing.assert_array_equal(out[i], oi[0])
        np.testing.assert_array_equal(dv[i], dvi[0])
        np.testing.assert_array_equal(df[i], dfi[0])


# --------------------------------------------------------------------------
# The quantity the lattice approximates (eq. 4-5): exact Gaussian filtering
# --------------------------------------------------------------------------

def test_against_exact_gaussian_12cube(O, capsys):
    """12^3 corner of the 32^3, d=3 workload (N = 1728), fp64 brute force.
    The lattice is an approximation: the errors are reported, and only
    flagged when far outside what a unit-variance lattice filter gives."""
    data = synth.generate("C1", shape=(12, 12, 12))
    f, v = data["f"], data["v"].astype(np.float64)
    lat = O.lattice(f)
    exact = O.gauss_bruteforce(f, v)
    exact_norm = exact / O.gauss_bruteforce(f, np.ones((f.shape[0], 1)))
    raw, _ = O.forward(lat, v, False)
    nrm, _ = O.forward(lat, v, True)
    err_raw = rel(raw, exact)
    err_norm = rel(nrm, exact_norm)
    gfit = float((raw * exact).sum() / (exact * exact).sum())
    with capsys.disabled():
        print(f"\n[approximation] 12^3 d=3: rel L2 raw {err_raw:.4f}, normalised {err_norm:.4f}, "
              f"gain fit/G_d {gfit:.4f}, M = {lat.M}")
    assert err_norm < 0.3
    assert err_raw < 0.3
    assert 0.8 < gfit < 1.25


@pytest.mark.parametrize("d", [2, 3])
def test_impulse_response_mass_and_variance(O, d, capsys):
    """One unit source among dense zero-valued probes: the raw response
    integrates to the Gaussian mass (2 pi)^{d/2} (pins s_d) and has unit
    second moment per input dimension (pins alpha)."""
    h = 0.2 if d == 2 else 0.3
    ext = 6.0 if d == 2 else 5.1
    axis = np.arange(-ext, ext + 1e-9, h)
    grid = np.stack(np.meshgrid(*([axis] * d), indexing="ij"), axis=-1).reshape(-1, d)
    src = np.array([[0.137, -0.071, 0.05][:d]])
    pts = np.concatenate([src, grid + 1e-3]).astype(np.float32)
    v = np.zeros((pts.shape[0], 1))
    v[0, 0] = 1.0
    lat = O.lattice(pts)
    out, _ = O.forward(lat, v, False)
    w = out[1:, 0]
    q = pts[1:].astype(np.float64) - pts[0].astype(np.float64)
    mass = w.sum() * h ** d
    mean = (w[:, None] * q).sum(axis=0) / w.sum()
    var = (w[:, None] * (q - mean) ** 2).sum(axis=0) / w.sum()
    with capsys.disabled():
        print(f"\n[impulse d={d}] mass/(2pi)^(d/2) = {mass / (2 * math.pi) ** (d / 2):.4f}, "
              f"mean {np.round(mean, 4)}, var {np.round(var, 4)}")
    assert mass == pytest.approx((2 * math.pi) ** (d / 2), rel=0.02)
    assert np.all(np.abs(mean) < 0.05)
    assert np.all(np.abs(var - 1.0) < 0.12)


# --------------------------------------------------------------------------
# Exact identities of the filter
# --------------------------------------------------------------------------

def cloud(d, n, s, scale=5.0):
    rng = np.random.default_rng(s)
    f = rng.uniform(0, scale, size=(n, d)).astype(np.float32)
    return f, rng


@pytest.mark.parametrize("d", [2, 3, 5])
def test_normalised_constant_survives(O, d):
    f, _ = cloud(d, 800, 600 + d)
    lat = O.lattice(f)
    out, _ = O.forward(lat, np.full((f.shape[0], 2), 3.7), True)
    np.testing.assert_allclose(out, 3.7, rtol=1e-12)


@pytest.mark.parametrize("normalize", [False, True])
def test_linearity(O, normalize):
    f, rng = cloud(3, 700, 700)
    lat = O.lattice(f)
    v1 = rng.standard_normal((700, 3))
    v2 = rng.standard_normal((700, 3))
    a, b = 1.7, -0.3
    o12, _ = O.forward(lat, a * v1 + b * v2, normalize)
    o1, _ = O.forward(lat, v1, normalize)
    o2, _ = O.forward(lat, v2, normalize)
    np.testing.assert_allclose(o12, a * o1 + b * o2, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("d", [2, 3, 5])
@pytest.mark.parametrize("normalize", [False, True])
def test_value_gradient_is_adjoint(O, d, normalize):
    """Eq. (7): <g, fwd(v)> = <dL/dv(g), v>, which holds only if the
    backward blur runs the directions in reverse order."""
    f, rng = cloud(d, 900, 800 + d, scale=3.0)
    lat = O.lattice(f)
    v = rng.standard_normal((900, 4))
    g = rng.standard_normal((900, 4))
    out, st = O.forward(lat, v, normalize)
    dv, _ = O.backward(lat, v, g, normalize, st)
    lhs = float((g * out).sum())
    rhs = float((dv * v).sum())
    assert lhs == pytest.approx(rhs, rel=1e-12)


def loss(O, f, v, g, normalize):
    lat = O.lattice(f)
    out, _ = O.forward(lat, v, normalize)
    return float((g * out).sum()), lat


@pytest.mark.parametrize("d", [2, 3, 5])
@pytest.mark.parametrize("normalize", [False, True])
def test_embedding_gradient_finite_differences(O, d, normalize):
    """Eq. (8) against central differences of L = <g, v'> in f, taken only
    where the point's simplex does not change.  In raw mode L is quadratic
    in f_i inside a simplex, so the difference quotient is exact."""
    n = 300
    f, rng = cloud(d, n, 900 + d, scale=2.5)
    v = rng.standard_normal((n, 3))
    g = rng.standard_normal((n, 3))
    L0, lat = loss(O, f, v, g, normalize)
    _, st = O.forward(lat, v, normalize)
    _, df = O.backward(lat, v, g, normalize, st)
    step = 2e-3 if normalize else 1e-2
    checked = 0
    for i in rng.choice(n, size=12, replace=False):
        for c in range(d):
            fp, fm = f.copy(), f.copy()
            fp[i, c] = np.float32(f[i, c] + step)
            fm[i, c] = np.float32(f[i, c] - step)
            s0, sp, sm = (O.simplex(x[i:i + 1]) for x in (f, fp, fm))
            if not (np.array_equal(sp.keys, s0.keys) and np.array_equal(sm.keys, s0.keys)
                    and np.array_equal(sp.rank, s0.rank) and np.array_equal(sm.rank, s0.rank)):
                continue
            Lp, _ = loss(O, fp, v, g, normalize)
            Lm, _ = loss(O, fm, v, g, normalize)
            fd = (Lp - Lm) / (float(fp[i, c]) - float(fm[i, c]))
            tol = (1e-4 if normalize else 1e-8) * (1.0 + abs(df[i, c]))
            assert abs(fd - df[i, c]) < tol, (i, c, fd, df[i, c])
            checked += 1
    assert checked >= 10


@pytest.mark.parametrize("d", [3, 5])
def test_translation_by_lattice_vector(O, d):
    """Shifting every point by t with E t = (d+1) z (z integer, sum 0)
    shifts every key by (d+1) z and leaves the output unchanged."""
    f, rng = cloud(d, 600, 1000 + d, scale=4.0)
    v = rng.standard_normal((600, 2))
    z = np.zeros(d + 1)
    z[0], z[2] = 1, -1
    E = O.embedding_matrix(d)
    t = E.T @ ((d + 1) * z) / O.alpha(d) ** 2
    np.testing.assert_allclose(E @ t, (d + 1) * z, atol=1e-12)
    f2 = (f.astype(np.float64) + t).astype(np.float32)
    lat1, lat2 = O.lattice(f), O.lattice(f2)
    K1 = full_keys(lat1.simp.keys.astype(np.int64))
    K2 = full_keys(lat2.simp.keys.astype(np.int64))
    same = np.all(K2 == K1 + ((d + 1) * z).astype(np.int64), axis=(1, 2))
    assert same.mean() > 0.99
    o1, _ = O.forward(lat1, v, False)
    o2, _ = O.forward(lat2, v, False)
    if same.all():
        np.testing.assert_allclose(o2, o1, rtol=1e-5, atol=1e-6 * np.abs(o1).max())


# --------------------------------------------------------------------------
# Planted mistakes: each must be caught by one of the pins above
# --------------------------------------------------------------------------

def test_planted_forward_order_in_backward_breaks_adjoint(O):
    f, rng = cloud(3, 900, 1103, scale=3.0)
    lat = O.lattice(f)
    v = rng.standard_normal((900, 2))
    g = rng.standard_normal((900, 2))
    out, st = O.forward(lat, v, False)
    wrong = O.raw_scale(3) * O.slice_(lat, O.blur(lat, O.splat(lat, g), reverse=False))
    lhs = float((g * out).sum())
    assert abs(lhs - float((wrong * v).sum())) > 1e-9 * abs(lhs)


def test_planted_missing_blur_term_breaks_textbook(O):
    rng = np.random.default_rng(12)
    p = rng.uniform(0, 4, 30).astype(np.float32)
    v = rng.standard_normal((30, 1))
    lat = O.lattice(p.reshape(-1, 1))
    A = O.splat(lat, v)
    # a single blur pass instead of d+1 = 2
    one = A.copy()
    for m in range(lat.M):
        lo, hi = lat.nbr[m, 0]
        one[m] = 2 * A[m] + (A[lo] if lo >= 0 else 0) + (A[hi] if hi >= 0 else 0)
    wrong = O.raw_scale(1) * O.slice_(lat, one)
    assert rel(wrong, textbook_1d(p.astype(np.float64), v, False)) > 0.1


def test_planted_dropped_gradient_term_breaks_finite_differences(O):
    d, n = 3, 200
    f, rng = cloud(d, n, 1200, scale=2.0)
    v = rng.standard_normal((n, 2))
    g = rng.standard_normal((n, 2))
    _, lat = loss(O, f, v, g, False)
    out, st = O.forward(lat, v, False)
    s = O.raw_scale(d)
    # keep only the slice term of eq. (8), drop the splat term
    df_wrong = O.embed_grad(lat, s * O.vertex_dots(lat, g, st["A"]))
    _, df = O.backward(lat, v, g, False, st)
    i, c = 5, 1
    fp, fm = f.copy(), f.copy()
    fp[i, c] += np.float32(1e-2)
    fm[i, c] -= np.float32(1e-2)
    Lp, _ = loss(O, fp, v, g, False)
    Lm, _ = loss(O, fm, v, g, False)
    fd = (Lp - Lm) / (float(fp[i, c]) - float(fm[i, c]))
    assert abs(fd - df[i, c]) < 1e-8 * (1 + abs(fd))
    assert abs(fd - df_wrong[i, c]) > 1e-3 * (1 + abs(fd))


# --------------------------------------------------------------------------
# Augmented-channel embedding gradient (the gradient of the exact Gaussian
# sum written with filters of the products f (x) v and f (x) g, each filter
# then replaced by the lattice one)
# --------------------------------------------------------------------------

def gauss_loss_fd(O, p, v, g, h=1e-5):
    """Central finite differences of L(p) = sum_i <g_i, sum_j exp(-|p_i-p_j|^2/2) v_j>."""
    fd = np.zeros_like(p)
    for i in range(p.shape[0]):
        for a in range(p.shape[1]):
            pp = p.copy()
            pp[i, a] += h
            lp = float((g * O.gauss_bruteforce(pp, v)).sum())
            pp[i, a] -= 2 * h
            lm = float((g * O.gauss_bruteforce(pp, v)).sum())
            fd[i, a] = (lp - lm) / (2 * h)
    return fd


@pytest.mark.parametrize("d", [1, 2, 3, 5])
def test_augmented_formula_is_exact_for_the_gaussian(O, d):
    """With the exact Gaussian as the filter the augmented-channel formula
    is the gradient of the Gaussian loss: finite differences, fp64."""
    rng = np.random.default_rng(1300 + d)
    n = 36
    p = rng.uniform(0, 2.5, (n, d))
    v = rng.standard_normal((n, 3))
    g = rng.standard_normal((n, 3))
    gr = O.egrad_exact_gaussian(p, v, g)
    fd = gauss_loss_fd(O, p, v, g)
    assert np.abs(gr - fd).max() < 1e-7 * max(1.0, np.abs(fd).max())


def test_augmented_gradient_against_exact_gaussian_12cube(O, capsys):
    """12^3 corner of the 32^3, d=3 workload: the lattice estimate of the
    augmented-channel gradient against the exact Gaussian gradient (the
    stated approximation error), next to the eq. 8 gradient, which is the
    derivative of the lattice output with the simplices held fixed."""
    data = synth.generate("C1", shape=(12, 12, 12))
    f = data["f"]
    v, g = data["v"].astype(np.float64), data["g"].astype(np.float64)
    lat = O.lattice(f)
    exact = O.egrad_exact_gaussian(f, v, g)
    aug = O.backward_augmented(lat, f, v, g)
    _, eq8 = O.backward(lat, v, g, False)
    err_aug, err_eq8 = rel(aug, exact), rel(eq8, exact)
    with capsys.disabled():
        print(f"\n[approximation] 12^3 d=3 embedding gradient vs exact Gaussian: rel L2 augmented {err_aug:.4f}, "
              f"eq. 8 {err_eq8:.4f}")
    assert err_aug < 0.35
    assert err_aug < err_eq8


@pytest.mark.parametrize("d", [3, 5])
def test_augmented_gradient_translation_by_lattice_vector(O, d):
    """A shift t by a lattice vector leaves the lattice filter unchanged,
    and W((p+t) (x) v) = W(p (x) v) + t (x) W v cancels against the
    -(p+t) W v terms: the estimate is unchanged."""
    f, rng = cloud(d, 500, 1400 + d, scale=4.0)
    v = rng.standard_normal((500, 3))
    g = rng.standard_normal((500, 3))
    z = np.zeros(d + 1)
    z[1], z[3] = 1, -1
    E = O.embedding_matrix(d)
    t = E.T @ ((d + 1) * z) / O.alpha(d) ** 2
    f2 = (f.astype(np.float64) + t).astype(np.float32)
    lat1, lat2 = O.lattice(f), O.lattice(f2)
    K1 = full_keys(lat1.simp.keys.astype(np.int64))
    K2 = full_keys(lat2.simp.keys.astype(np.int64))
    if not np.all(K2 == K1 + ((d + 1) * z).astype(np.int64)):
        pytest.skip("a rank tie changed under the shift")
    a1 = O.backward_augmented(lat1, f, v, g)
    a2 = O.backward_augmented(lat2, f2, v, g)
    assert rel(a2, a1) < 1e-5  # fp32 shifted features perturb the weights slightly


def test_planted_dropped_receiver_term_breaks_augmented_pins(O):
    """Dropping the -p_i (W v)_i term breaks both the finite-difference
    reduction and the translation invariance."""
    rng = np.random.default_rng(1500)
    n, d = 30, 2
    p = rng.uniform(0, 2.5, (n, d))
    v = rng.standard_normal((n, 2))
    g = rng.standard_normal((n, 2))

    def K(x):
        return O.gauss_bruteforce(p, x)

    Wpv = K(O.augmented_channels(p, v)).reshape(n, d, 2)
    Wpg = K(O.augmented_channels(p, g)).reshape(n, d, 2)
    wrong = (np.einsum("nac,nc->na", Wpv, g) + np.einsum("nac,nc->na", Wpg, v)
             - p * (v * K(g)).sum(axis=1, keepdims=True))
    fd = gauss_loss_fd(O, p, v, g)
    assert np.abs(wrong - fd).max() > 1e-3 * np.abs(fd).max()


# --------------------------------------------------------------------------
# Asymmetric filter: values splatted at the keys, read at the queries, over
# the lattice of [keys; queries]
# --------------------------------------------------------------------------

def asym_case(d, nk, nq, seed, shift=0.37):
    rng = np.random.default_rng(seed)
    k = rng.uniform(0, 4.0, (nk, d)).astype(np.float32)
    q = (rng.uniform(0, 4.0, (nq, d)) + shift).astype(np.float32)
    v = rng.standard_normal((nk, 3))
    g = rng.standard_normal((nq, 3))
    return k, q, v, g


def test_asym_against_exact_gaussian_12cube(O, capsys):
    """Keys: the 12^3 corner of the 32^3 d=3 workload; queries: the same
    voxels moved by half a voxel along each axis.  Stated approximation
    error against the exact sum_j exp(-|q_i - k_j|^2/2) v_j."""
    data = synth.generate("C1", shape=(12, 12, 12))
    k = data["f"]
    q = (k.astype(np.float64) + 0.5 / 4.0).astype(np.float32)
    v = data["v"].astype(np.float64)
    lat = O.lattice(np.concatenate([k, q]))
    out, _ = O.forward_asym(lat, k.shape[0], v)
    exact = O.gauss_bruteforce_asym(q, k, v)
    err = rel(out, exact)
    with capsys.disabled():
        print(f"\n[approximation] asymmetric 12^3 d=3, queries moved by half a voxel: rel L2 {err:.4f}")
    assert err < 0.3


@pytest.mark.parametrize("d", [2, 3, 5])
def test_asym_value_gradient_is_adjoint(O, d):
    """<g, out(v)> = <dL/dv(g), v>: the query gradients are splatted at the
    queries and read at the keys."""
    k, q, v, g = asym_case(d, 700, 500, 1800 + d)
    lat = O.lattice(np.concatenate([k, q]))
    out, st = O.forward_asym(lat, 700, v)
    dv, _ = O.backward_asym(lat, 700, v, g, st)
    assert float((g * out).sum()) == pytest.approx(float((dv * v).sum()), rel=1e-12)


def test_asym_queries_equal_to_keys_is_the_symmetric_filter(O):
    """With q = k the output is the symmetric filter's, dL/dv too, and the
    key and query rows of dL/df add up to the symmetric gradient."""
    f, rng = cloud(3, 600, 1900, scale=3.0)
    v = rng.standard_normal((600, 2))
    g = rng.standard_normal((600, 2))
    sym = O.lattice(f)
    o_s, st_s = O.forward(sym, v, False)
    dv_s, df_s = O.backward(sym, v, g, False, st_s)
    lat = O.lattice(np.concatenate([f, f]))
    assert lat.M == sym.M
    o_a, st = O.forward_asym(lat, 600, v)
    dv_a, df_a = O.backward_asym(lat, 600, v, g, st)
    np.testing.assert_allclose(o_a, o_s, rtol=1e-11, atol=1e-12 * np.abs(o_s).max())
    np.testing.assert_allclose(dv_a, dv_s, rtol=1e-11, atol=1e-12 * np.abs(dv_s).max())
    np.testing.assert_allclose(df_a[:600] + df_a[600:], df_s, rtol=1e-10, atol=1e-11 * np.abs(df_s).max())


@pytest.mark.parametrize("d", [2, 3])
def test_asym_embedding_gradient_finite_differences(O, d):
    """Central differences of L = <g, out> with respect to key and query
    coordinates, where the perturbation keeps every simplex (L is then
    quadratic in the moved point, so central differences are exact)."""
    k, q, v, g = asym_case(d, 300, 200, 2000 + d)
    nk = k.shape[0]
    pts = np.concatenate([k, q])

    def L(p):
        lat = O.lattice(p)
        out, _ = O.forward_asym(lat, nk, v)
        return float((g * out).sum()), lat

    _, lat = L(pts)
    _, df = O.backward_asym(lat, nk, v, g)
    checked = 0
    for i in (3, 17, 250, nk + 5, nk + 120):
        for c in range(d):
            h = np.float32(1e-2)
            pp, pm = pts.copy(), pts.copy()
            pp[i, c] += h
            pm[i, c] -= h
            Lp, lp = L(pp)
            Lm, lm = L(pm)
            same = (np.array_equal(lp.simp.keys, lat.simp.keys) and np.array_equal(lm.simp.keys, lat.simp.keys)
                    and np.array_equal(lp.simp.rank, lat.simp.rank) and np.array_equal(lm.simp.rank, lat.simp.rank))
            if not same:
                continue
            fd = (Lp - Lm) / (float(pp[i, c]) - float(pm[i, c]))
            assert abs(fd - df[i, c]) < 1e-8 * (1 + abs(fd))
            checked += 1
    assert checked >= 4


def test_filter_at_points_equals_the_whole_filter(O):
    """The per-point evaluation used by the sampled full-size parity tests
    gives the whole-volume result at those points."""
    f, rng = cloud(4, 900, 2500, scale=3.0)
    v = rng.standard_normal((900, 3))
    g = rng.standard_normal((900, 3))
    lat = O.lattice(f)
    out, st = O.forward(lat, v, False)
    dv, df = O.backward(lat, v, g, False, st)
    idx = np.sort(rng.choice(900, 200, replace=False))
    o2, dv2, df2 = O.filter_at(lat, v, g, idx)
    np.testing.assert_allclose(o2, out[idx], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dv2, dv[idx], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(df2, df[idx], rtol=1e-12, atol=1e-14)
