"""Parity of the permutohedral-block prologue (pam_block_fwd / _bwd, through
the C ABI) with the oracle, and of the whole block: prologue, batched
lattice build over the channel groups, filter, backward, prologue
backward."""
import numpy as np
import pytest

from helpers import log, rel_l2, row_errors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1907_00641_amd.binding as B

    B.lib()


def params(c_in, d_tot, c_tot, dims, seed):
    rng = np.random.default_rng(seed)
    n = dims[0] * dims[1] * dims[2]
    x = rng.standard_normal((n, c_in)).astype(np.float32)
    wf = (rng.standard_normal((d_tot, c_in + 3)) / np.sqrt(c_in + 3)).astype(np.float32)
    bf = (0.1 * rng.standard_normal(d_tot)).astype(np.float32)
    wv = (rng.standard_normal((c_tot, c_in)) / np.sqrt(c_in)).astype(np.float32)
    bv = (0.1 * rng.standard_normal(c_tot)).astype(np.float32)
    return x, wf, bf, wv, bv


CASES = [(18, 10, 16, 2, (9, 7, 5)), (5, 3, 7, 1, (13, 11, 3)), (64, 32, 128, 2, (4, 4, 4)), (7, 16, 24, 8, (33, 2, 2))]


@pytest.mark.parametrize("c_in,d_tot,c_tot,groups,dims", CASES, ids=["c18d10v16g2", "c5d3v7g1", "limits", "g8"])
def test_prologue_matches_oracle(c_in, d_tot, c_tot, groups, dims):
    import torch

    import paper_1907_00641_amd as P
    from oracle import block as OB

    x, wf, bf, wv, bv = params(c_in, d_tot, c_tot, dims, 3000 + c_in)
    log(f"[block] c_in={c_in} d_tot={d_tot} c_tot={c_tot} groups={groups} dims={dims}")
    dev = torch.device("cuda:0")
    T = [torch.from_numpy(a).to(dev) for a in (x, wf, bf, wv, bv)]
    desc = P.block_desc(c_in, d_tot, c_tot, groups, dims, 0.125, 0.05)
    feat, val = P.pam_block_fwd(desc, *T)
    f_o, v_o = OB.prologue_fwd(x, dims, wf, bf, wv, bv, 0.125, 0.05, groups)
    rng = np.random.default_rng(7)
    gf = rng.standard_normal(f_o.shape).astype(np.float32)
    gv = rng.standard_normal(v_o.shape).astype(np.float32)
    grads = P.pam_block_bwd(desc, T[0], T[1], T[2], T[3], torch.from_numpy(gf).to(dev), torch.from_numpy(gv).to(dev))
    torch.cuda.synchronize()
    g_o = OB.prologue_bwd(x, dims, wf, bf, wv, 0.125, 0.05, groups, gf, gv)
    assert rel_l2(feat.cpu().numpy(), f_o) < 1e-5
    assert rel_l2(val.cpu().numpy(), v_o) < 1e-5
    for name, a, b in zip(("dx", "dwf", "dbf", "dwv", "dbv"), grads, g_o):
        e = rel_l2(a.cpu().numpy(), b)
        log(f"  {name} rel L2 {e:.2e}")
        assert e < 1e-4, name


def test_prologue_argument_errors():
    import ctypes

    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    L = B.lib()
    dev = torch.device("cuda:0")
    buf = torch.zeros(1 << 16, device=dev)
    p = buf.data_ptr()
    bad = [P.block_desc(0, 4, 4, 1, (4, 4, 4), 1.0, 0.01), P.block_desc(65, 4, 4, 1, (4, 4, 4), 1.0, 0.01),
           P.block_desc(4, 5, 4, 2, (4, 4, 4), 1.0, 0.01), P.block_desc(4, 34, 4, 2, (4, 4, 4), 1.0, 0.01),
           P.block_desc(4, 4, 130, 2, (4, 4, 4), 1.0, 0.01), P.block_desc(4, 4, 4, 1, (0, 4, 4), 1.0, 0.01),
           P.block_desc(4, 17, 4, 1, (4, 4, 4), 1.0, 0.01)]
    for d in bad:
        assert L.pam_block_fwd(ctypes.byref(d), p, p, p, p, p, p + 4096, p + 65536,
                               None) == B.PAM_ERR_INVALID_ARGUMENT
        assert L.pam_block_bwd_workspace(ctypes.byref(d)) == 0
    good = P.block_desc(4, 4, 4, 2, (4, 4, 4), 1.0, 0.01)
    assert L.pam_block_fwd(ctypes.byref(good), p, p, p, p, p, None, p, None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_block_fwd(None, p, p, p, p, p, p, p, None) == B.PAM_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("dims,mesh_scale", [((12, 10, 8), 0.25), ((80, 80, 48), 1.0 / 8.0)],
                         ids=["12x10x8", "80x80x48"])
def test_block_end_to_end(O, dims, mesh_scale):
    """Prologue -> batched build over the two channel groups -> filter ->
    backward -> prologue backward, against the same chain on the oracle.
    80x80x48 with mesh scale 1/8 is the half-resolution shape the benchmark
    times (U-PAM-Net, 18 input channels, two groups of d = 5 and C = 8)."""
    import torch

    import paper_1907_00641_amd as P
    from oracle import block as OB

    c_in, d_tot, c_tot, G = 18, 10, 16, 2
    n = dims[0] * dims[1] * dims[2]
    log(f"[block e2e] dims={dims} n={n}")
    x, wf, bf, wv, bv = params(c_in, d_tot, c_tot, dims, 3100)
    rng = np.random.default_rng(3101)
    gout = rng.standard_normal((G * n, c_tot // G)).astype(np.float32)
    dev = torch.device("cuda:0")
    T = [torch.from_numpy(a).to(dev) for a in (x, wf, bf, wv, bv)]
    desc = P.block_desc(c_in, d_tot, c_tot, G, dims, mesh_scale, 0.01)
    feat, val = P.pam_block_fwd(desc, *T)
    lat = P.pam_lattice_build(feat, group_start=[0, n, 2 * n])
    out = P.pam_filter_fwd(lat, val)
    dval, dfeat = P.pam_filter_bwd(lat, val, torch.from_numpy(gout).to(dev))
    grads = P.pam_block_bwd(desc, T[0], T[1], T[2], T[3], dfeat, dval)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    grads = [g.cpu().numpy() for g in grads]
    lat.destroy()
    # the oracle chain: each group's lattice on its own
    f_o, v_o = OB.prologue_fwd(x, dims, wf, bf, wv, bv, mesh_scale, 0.01, G)
    f32 = f_o.astype(np.float32)
    out_o = np.zeros_like(v_o)
    df_o = np.zeros_like(f_o)
    dv_o = np.zeros_like(v_o)
    for g in range(G):
        s = slice(g * n, (g + 1) * n)
        olat = O.lattice(f32[s])
        o, st = O.forward(olat, v_o[s], False)
        dv, df = O.backward(olat, v_o[s], gout[s].astype(np.float64), False, st)
        out_o[s], dv_o[s], df_o[s] = o, dv, df
    g_o = OB.prologue_bwd(x, dims, wf, bf, wv, mesh_scale, 0.01, G, df_o, dv_o)
    errs = [rel_l2(out, out_o)] + [rel_l2(a, b) for a, b in zip(grads, g_o)]
    log(f"  rel L2 out {errs[0]:.2e} dx {errs[1]:.2e} dwf {errs[2]:.2e} dbf {errs[3]:.2e} "
        f"dwv {errs[4]:.2e} dbv {errs[5]:.2e}")
    assert max(errs) < 1e-4
    # per row: the output everywhere; dx where no pre-activation of the
    # voxel lies within 1e-5 of the Leaky-ReLU kink (there the fp32 GPU and
    # the fp64 oracle may legitimately take different slopes)
    z = np.concatenate([x.astype(np.float64), OB.mesh(dims, mesh_scale)], axis=1) @ wf.T.astype(np.float64) + bf
    smooth = np.abs(z).min(axis=1) > 1e-5
    log(f"  {int((~smooth).sum())} voxels with a pre-activation within 1e-5 of the kink")
    for name, a, b in (("out", out, out_o), ("dx", grads[0][smooth], g_o[0][smooth])):
        ratio, row, rerr = row_errors(a, b)
        log(f"  {name} worst row {row}: {rerr:.1e} of its norm, {ratio:.2f} of its bound")
        assert ratio <= 1.0, name
