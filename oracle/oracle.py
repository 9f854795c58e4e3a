"""Python face of the CPU oracle (``pam_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
CPU-baseline leg of the benchmark, never by the GPU library or its binding.

The C file holds the per-step loops; this module composes them in the
order the paper gives:

* forward, eq. (6):  v' = Sl(B(S(E(f), v)), E(f));
* value gradient, eq. (7): dL/dv = Sl(B~(S(E(f), dL/dv')), E(f)), where B~
  runs the blur directions in reverse order;
* embedding gradient, eq. (8): for each point, the blurred lattices of v
  (forward order) and of dL/dv' (reverse order) read at the point's simplex
  vertices, contracted with v_i and dL/dv'_i, combined through the
  permutation found by E and mapped back by E^T;
* asymmetric filter (raw mode): the same operators over the points
  [keys; queries] with the values carried by the keys only and the result
  read at the queries;
* augmented-channel embedding gradient (raw mode): the gradient of the
  exact Gaussian sum written with filters of the products f (x) v and
  f (x) dL/dv', each filter then replaced by the lattice one.

Two output modes.  ``normalize=False`` (raw) scales the sliced result by
s_d = 1/G_d so that it approximates sum_j exp(-|f_i-f_j|^2/2) v_j;
``normalize=True`` divides by the same filter applied to a constant-1
channel (the normalised non-local means form).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pam_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_ptr = ctypes.c_void_p


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2, no FMA contraction)."""
    stale = (not os.path.exists(_LIB)) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)
    if force or stale:
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-D_GNU_SOURCE", "-ffp-contract=off",
                               "-fno-fast-math", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        L.orc_alpha.restype = ctypes.c_double
        L.orc_alpha.argtypes = [ctypes.c_int]
        L.orc_raw_scale.restype = ctypes.c_double
        L.orc_raw_scale.argtypes = [ctypes.c_int]
        L.orc_embedding_matrix.argtypes = [ctypes.c_int, _ptr]
        L.orc_simplex.restype = ctypes.c_int
        L.orc_simplex.argtypes = [_ptr, _i64, ctypes.c_int, _ptr, _ptr, _ptr, _ptr]
        L.orc_lattice.restype = _i64
        L.orc_lattice.argtypes = [_i64, ctypes.c_int, _ptr, _ptr, _ptr]
        L.orc_neighbours.argtypes = [_i64, ctypes.c_int, _ptr, _ptr]
        L.orc_splat.argtypes = [_i64, ctypes.c_int, ctypes.c_int, _ptr, _ptr, _ptr, _i64, _ptr]
        L.orc_blur.restype = ctypes.c_int
        L.orc_blur.argtypes = [_i64, ctypes.c_int, ctypes.c_int, _ptr, ctypes.c_int, _ptr]
        L.orc_slice.argtypes = [_i64, ctypes.c_int, ctypes.c_int, _ptr, _ptr, _ptr, _ptr]
        L.orc_vertex_dots.argtypes = [_i64, ctypes.c_int, ctypes.c_int, _ptr, _ptr, _ptr, _ptr]
        L.orc_embed_grad.argtypes = [_i64, ctypes.c_int, _ptr, _ptr, _ptr]
        L.orc_gauss_bruteforce.argtypes = [_i64, ctypes.c_int, ctypes.c_int, _ptr, _ptr, _ptr]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def alpha(d: int) -> float:
    return lib().orc_alpha(d)


def raw_scale(d: int) -> float:
    return lib().orc_raw_scale(d)


def embedding_matrix(d: int) -> np.ndarray:
    E = np.zeros((d + 1, d), dtype=np.float64)
    lib().orc_embedding_matrix(d, _p(E))
    return E


@dataclass
class Simplices:
    keys: np.ndarray   # n x (d+1) x d int32
    bary: np.ndarray   # n x (d+1) fp64
    rank: np.ndarray   # n x (d+1) int32
    xelev: np.ndarray  # n x (d+1) fp64


def simplex(f: np.ndarray) -> Simplices:
    """Operator E: enclosing simplex of every point of f (n x d fp32)."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    n, d = f.shape
    keys = np.zeros((n, d + 1, d), dtype=np.int32)
    bary = np.zeros((n, d + 1), dtype=np.float64)
    rank = np.zeros((n, d + 1), dtype=np.int32)
    xel = np.zeros((n, d + 1), dtype=np.float64)
    rc = lib().orc_simplex(_p(f), n, d, _p(keys), _p(bary), _p(rank), _p(xel))
    if rc != 0:
        raise ValueError("embedding out of the representable key range")
    return Simplices(keys, bary, rank, xel)


@dataclass
class Lattice:
    d: int
    simp: Simplices
    vert: np.ndarray   # n x (d+1) int32 vertex ids (lexicographic key order)
    keys: np.ndarray   # M x d int32, sorted
    nbr: np.ndarray    # M x (d+1) x 2 int32; [...,0] = key - u_j, [...,1] = key + u_j

    @property
    def M(self) -> int:
        return self.keys.shape[0]

    @property
    def n(self) -> int:
        return self.vert.shape[0]


def lattice(f: np.ndarray) -> Lattice:
    """Embedding plus the sparse lattice (vertex set, ids, neighbours)."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    n, d = f.shape
    s = simplex(f)
    vert = np.zeros((n, d + 1), dtype=np.int32)
    ukeys = np.zeros((max(n * (d + 1), 1), d), dtype=np.int32)
    M = lib().orc_lattice(n, d, _p(s.keys), _p(vert), _p(ukeys))
    if M < 0:
        raise MemoryError("oracle lattice build")
    ukeys = np.ascontiguousarray(ukeys[:M])
    nbr = np.zeros((M, d + 1, 2), dtype=np.int32)
    lib().orc_neighbours(M, d, _p(ukeys), _p(nbr))
    return Lattice(d, s, vert, ukeys, nbr)


def splat(lat: Lattice, val: np.ndarray) -> np.ndarray:
    val = np.ascontiguousarray(val, dtype=np.float64)
    C = val.shape[1]
    L = np.zeros((lat.M, C), dtype=np.float64)
    lib().orc_splat(lat.n, lat.d, C, _p(lat.vert), _p(lat.simp.bary), _p(val), lat.M, _p(L))
    return L


def blur(lat: Lattice, L: np.ndarray, reverse: bool) -> np.ndarray:
    L = np.array(L, dtype=np.float64, order="C", copy=True)
    if lib().orc_blur(lat.M, lat.d, L.shape[1], _p(lat.nbr), int(reverse), _p(L)) != 0:
        raise MemoryError("oracle blur")
    return L


def slice_(lat: Lattice, L: np.ndarray) -> np.ndarray:
    L = np.ascontiguousarray(L, dtype=np.float64)
    C = L.shape[1]
    out = np.zeros((lat.n, C), dtype=np.float64)
    lib().orc_slice(lat.n, lat.d, C, _p(lat.vert), _p(lat.simp.bary), _p(L), _p(out))
    return out


def vertex_dots(lat: Lattice, a: np.ndarray, L: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float64)
    L = np.ascontiguousarray(L, dtype=np.float64)
    h = np.zeros((lat.n, lat.d + 1), dtype=np.float64)
    lib().orc_vertex_dots(lat.n, lat.d, a.shape[1], _p(lat.vert), _p(a), _p(L), _p(h))
    return h


def embed_grad(lat: Lattice, h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.float64)
    df = np.zeros((lat.n, lat.d), dtype=np.float64)
    lib().orc_embed_grad(lat.n, lat.d, _p(lat.simp.rank), _p(h), _p(df))
    return df


def _ones(lat: Lattice) -> np.ndarray:
    return np.ones((lat.n, 1), dtype=np.float64)


def forward(lat: Lattice, v: np.ndarray, normalize: bool = False):
    """Eq. (6).  Returns (out, state) where state keeps the blurred lattices
    for the backward pass."""
    A = blur(lat, splat(lat, v), reverse=False)
    if normalize:
        Aw = blur(lat, splat(lat, _ones(lat)), reverse=False)
        num = slice_(lat, A)
        z = slice_(lat, Aw)
        out = num / z
        return out, {"A": A, "Aw": Aw, "z": z, "out": out}
    out = raw_scale(lat.d) * slice_(lat, A)
    return out, {"A": A, "out": out}


def backward(lat: Lattice, v: np.ndarray, g: np.ndarray, normalize: bool = False, state=None):
    """Eq. (7) for dL/dv and eq. (8) for dL/df.  Returns (dv, df)."""
    v = np.asarray(v, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    if state is None:
        _, state = forward(lat, v, normalize)
    A = state["A"]
    if not normalize:
        s = raw_scale(lat.d)
        At = blur(lat, splat(lat, g), reverse=True)
        dv = s * slice_(lat, At)
        h = s * (vertex_dots(lat, g, A) + vertex_dots(lat, v, At))
        return dv, embed_grad(lat, h)
    # normalised mode: out = N / z with N = Sl B S v and z = Sl B S 1.
    # dL/dN_i = g_i / z_i, dL/dz_i = -<g_i, out_i> / z_i (quotient rule).
    Aw, z, out = state["Aw"], state["z"], state["out"]
    gt = g / z
    gam = -(g * out).sum(axis=1, keepdims=True) / z
    At = blur(lat, splat(lat, gt), reverse=True)
    Atw = blur(lat, splat(lat, gam), reverse=True)
    dv = slice_(lat, At)
    h = (vertex_dots(lat, gt, A) + gam * Aw[lat.vert, 0]
         + vertex_dots(lat, v, At) + Atw[lat.vert, 0])
    return dv, embed_grad(lat, h)


def gauss_bruteforce(p: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Exact sum_j exp(-|p_i - p_j|^2/2) v_j in fp64, O(n^2)."""
    p = np.ascontiguousarray(p, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    n, d = p.shape
    out = np.zeros((n, v.shape[1]), dtype=np.float64)
    lib().orc_gauss_bruteforce(n, d, v.shape[1], _p(p), _p(v), _p(out))
    return out


def augmented_channels(p: np.ndarray, x: np.ndarray) -> np.ndarray:
    """n x (d*C) columns; column a*C + c holds p_a * x_c."""
    p = np.asarray(p, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    n, d = p.shape
    return (p[:, :, None] * x[:, None, :]).reshape(n, d * x.shape[1])


def egrad_from_filters(W, Wt, p: np.ndarray, v: np.ndarray, g: np.ndarray) -> np.ndarray:
    """dL/dp for L = sum_i <g_i, (W v)_i> when W has the Gaussian weights
    K_ij = exp(-|p_i - p_j|^2 / 2) (eq. 4-5 as read here).  Since
    dK_ij/dp_i = (p_j - p_i) K_ij, the point i gets
        sum_c g_ic [W(p (x) v)_ic - p_i (W v)_ic]      (i as the receiving point)
      + sum_c v_ic [W^T(p (x) g)_ic - p_i (W^T g)_ic]  (i as a source point),
    where W(p (x) v)_ic is the d-vector sum_j K_ij p_j v_jc.  W and Wt apply
    the filter and its transpose to n x k arrays."""
    p = np.asarray(p, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    n, d = p.shape
    C = v.shape[1]
    Wv = W(v)
    Wtg = Wt(g)
    Wpv = W(augmented_channels(p, v)).reshape(n, d, C)
    Wtpg = Wt(augmented_channels(p, g)).reshape(n, d, C)
    recv = np.einsum("nac,nc->na", Wpv, g) - p * (g * Wv).sum(axis=1, keepdims=True)
    src = np.einsum("nac,nc->na", Wtpg, v) - p * (v * Wtg).sum(axis=1, keepdims=True)
    return recv + src


def backward_augmented(lat: Lattice, f: np.ndarray, v: np.ndarray, g: np.ndarray) -> np.ndarray:
    """Augmented-channel embedding gradient (raw mode): egrad_from_filters
    with W = s_d Sl B S (forward blur order) and its transpose
    W^T = s_d Sl B~ S (reversed order, as for eq. 7)."""
    s = raw_scale(lat.d)

    def W(x):
        return s * slice_(lat, blur(lat, splat(lat, x), reverse=False))

    def Wt(x):
        return s * slice_(lat, blur(lat, splat(lat, x), reverse=True))

    return egrad_from_filters(W, Wt, f, v, g)


def egrad_exact_gaussian(p: np.ndarray, v: np.ndarray, g: np.ndarray) -> np.ndarray:
    """The same formula with the exact O(n^2) Gaussian for W (= W^T)."""
    p = np.asarray(p, dtype=np.float64)

    def K(x):
        return gauss_bruteforce(p, x)

    return egrad_from_filters(K, K, p, v, g)


def forward_asym(lat: Lattice, n_keys: int, v: np.ndarray):
    """Asymmetric filter (raw mode) over the lattice of the points
    [keys; queries]: the key values are splatted (the queries carry none),
    the result is read at the queries.  Returns (out for the queries, state)."""
    v = np.asarray(v, dtype=np.float64)
    vu = np.zeros((lat.n, v.shape[1]), dtype=np.float64)
    vu[:n_keys] = v
    out, st = forward(lat, vu, False)
    st["vu"] = vu
    return out[n_keys:], st


def backward_asym(lat: Lattice, n_keys: int, v: np.ndarray, g: np.ndarray, state=None):
    """Backward pass of forward_asym: the query gradients are splatted (the
    keys carry none).  Returns (dL/dv for the keys, dL/df for all points)."""
    if state is None:
        _, state = forward_asym(lat, n_keys, v)
    g = np.asarray(g, dtype=np.float64)
    gu = np.zeros((lat.n, g.shape[1]), dtype=np.float64)
    gu[n_keys:] = g
    dv, df = backward(lat, state["vu"], gu, False, state)
    return dv[:n_keys], df


def gauss_bruteforce_asym(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Exact sum_j exp(-|q_i - k_j|^2/2) v_j in fp64, O(nq nk)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros((q.shape[0], v.shape[1]), dtype=np.float64)
    for i0 in range(0, q.shape[0], 512):
        d2 = ((q[i0:i0 + 512, None, :] - k[None, :, :]) ** 2).sum(axis=-1)
        out[i0:i0 + 512] = np.exp(-0.5 * d2) @ v
    return out


def subset(lat: Lattice, idx: np.ndarray) -> Lattice:
    """The same lattice (vertex set, ids, neighbours) seen from the points
    idx only: slice_, vertex_dots and embed_grad then work on those points."""
    s = lat.simp
    sub = Simplices(s.keys[idx], s.bary[idx], s.rank[idx], s.xelev[idx])
    return Lattice(lat.d, sub, lat.vert[idx], lat.keys, lat.nbr)


def filter_at(lat: Lattice, v: np.ndarray, g: np.ndarray, idx: np.ndarray):
    """Raw-mode out, dL/dv and dL/df (eq. 6-8) at the points idx only: the
    blurred lattices are global, the slices and eq. 8 are taken per point."""
    s = raw_scale(lat.d)
    A = blur(lat, splat(lat, v), reverse=False)
    At = blur(lat, splat(lat, g), reverse=True)
    sub = subset(lat, idx)
    v = np.asarray(v, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    out = s * slice_(sub, A)
    dv = s * slice_(sub, At)
    h = s * (vertex_dots(sub, g[idx], A) + vertex_dots(sub, v[idx], At))
    return out, dv, embed_grad(sub, h)
