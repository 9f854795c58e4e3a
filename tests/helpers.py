"""Shared helpers of the GPU parity tests: run the HIP path through the C
ABI, canonicalise its lattice, compare with the oracle."""
import sys

import numpy as np


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def gpu_run(f, v=None, g=None, flags=0, bwd=True, grad_val=True, grad_feat=True, group_start=None):
    """Build + fwd (+ bwd) on cuda:0 through the C ABI; returns host arrays.
    ``group_start`` makes it a batched build (also returns ``vgroup``)."""
    import torch

    import paper_1907_00641_amd as P

    dev = torch.device("cuda:0")
    ft = torch.from_numpy(np.ascontiguousarray(f, dtype=np.float32)).to(dev)
    res = {}
    lat = P.pam_lattice_build(ft, group_start=group_start)
    res["M"], res["cap"] = P.pam_lattice_stats(lat)
    if v is not None:
        vt = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).to(dev)
        res["out"] = P.pam_filter_fwd(lat, vt, flags).cpu().numpy()
        if bwd:
            gt = torch.from_numpy(np.ascontiguousarray(g, dtype=np.float32)).to(dev)
            dv, df = P.pam_filter_bwd(lat, vt, gt, flags, grad_val=grad_val, grad_feat=grad_feat)
            res["dv"] = None if dv is None else dv.cpu().numpy()
            res["df"] = None if df is None else df.cpu().numpy()
    torch.cuda.synchronize()
    res["keys"], res["vert"], res["bary"], res["nbr"] = P.pam_lattice_export(lat)
    if group_start is not None:
        res["vgroup"] = P.pam_lattice_export_groups(lat)
    lat.destroy()
    return res


def group_part(res, grp, start, end):
    """The lattice of group ``grp`` (points [start, end)) of a batched build,
    as a result of its own: its vertices renumbered in id order.  Fails if a
    point or a neighbour link of the group reaches another group's vertex."""
    vg = res["vgroup"]
    sel = np.flatnonzero(vg == grp)
    local = np.full(len(vg), -1, dtype=np.int64)
    local[sel] = np.arange(len(sel))
    vert = local[res["vert"][start:end]]
    assert (vert >= 0).all(), "a point uses a vertex of another group"
    nb = res["nbr"][sel].astype(np.int64)
    nbl = np.where(nb >= 0, local[np.maximum(nb, 0)], -1)
    assert ((nb < 0) | (nbl >= 0)).all(), "a blur link crosses groups"
    return {"M": len(sel), "keys": res["keys"][sel], "vert": vert, "nbr": nbl}


def canonical_perm(gpu_keys):
    """Map GPU vertex ids to lexicographic-order ids (the oracle's)."""
    M = gpu_keys.shape[0]
    order = np.lexsort(gpu_keys.T[::-1]) if M else np.zeros(0, dtype=np.int64)
    perm = np.empty(M, dtype=np.int64)
    perm[order] = np.arange(M)
    return order, perm


def assert_lattice_equal(res, olat):
    """Keys, vertex count, per-point vertex ids and neighbour table equal to
    the oracle's, bit for bit, after mapping GPU ids through the keys."""
    M = olat.M
    assert res["M"] == M, (res["M"], M)
    order, perm = canonical_perm(res["keys"])
    np.testing.assert_array_equal(res["keys"][order], olat.keys)
    np.testing.assert_array_equal(perm[res["vert"]], olat.vert)
    nb = res["nbr"].astype(np.int64)
    mapped = np.where(nb >= 0, perm[np.maximum(nb, 0)], -1)
    canon = np.empty_like(mapped)
    canon[perm] = mapped
    np.testing.assert_array_equal(canon, olat.nbr)


def assert_bary_close(res, olat):
    """Barycentric weights of the records the filter kernels read (exported
    through the sorted order) within 1e-6 absolute of the oracle's fp64
    weights, at every size: the GPU forms the residuals x - r in fp64, so
    their error does not grow with |x|; the fp32 steps after that round at
    about 1e-7."""
    np.testing.assert_allclose(res["bary"], olat.simp.bary, rtol=0, atol=1e-6)


def row_errors(got, want, rel=1e-3, abs_rms=1e-6, extra=None):
    """Per-row check beside the whole-array relative L2: for every row i,
    ||got_i - want_i|| <= rel * ||want_i|| + abs_rms * rms (+ extra_i), where
    rms is the root mean square of the rows' norms of ``want``.  Returns the
    largest ratio of a row's error to its bound, that row, and its error
    relative to the row norm (ratio <= 1 passes)."""
    got = np.asarray(got, dtype=np.float64).reshape(len(want), -1)
    want = np.asarray(want, dtype=np.float64).reshape(len(want), -1)
    if want.size == 0:
        return 0.0, -1, 0.0
    err = np.linalg.norm(got - want, axis=1)
    nrm = np.linalg.norm(want, axis=1)
    rms = float(np.sqrt(np.mean(nrm * nrm)))
    bound = rel * nrm + abs_rms * rms
    if extra is not None:
        bound = bound + np.asarray(extra, dtype=np.float64)
    ratio = np.divide(err, bound, out=np.where(err > 0, np.inf, 0.0), where=bound > 0)
    i = int(np.argmax(ratio))
    return float(ratio[i]), i, float(err[i] / nrm[i]) if nrm[i] > 0 else float(err[i])


def df_term_scale(f, v, g, out, dv):
    """Per point, the size of the terms that cancel in its embedding
    gradient: eq. 8 differences <g, A_k> - <g, A_k'> and <v, At_k> - <v, At_k'>
    (of the order |g| |out| + |v| |dv| once scaled like the filter), and the
    augmented estimator's f (x) v filter minus f times the filter of v (an
    extra factor |f|).  fp32 evaluation leaves an error of a few hundred
    unit roundoffs of this size where the difference itself is small, so
    the per-row df bound adds 1e-5 of it."""
    n = len(f)
    rn = lambda a: np.linalg.norm(np.asarray(a, dtype=np.float64).reshape(n, -1), axis=1)
    return (1.0 + rn(f)) * (rn(g) * rn(out) + rn(v) * rn(dv))
