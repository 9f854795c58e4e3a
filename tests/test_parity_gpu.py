"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bar: lattice keys, vertex count, per-point vertex ids and neighbour table
bit-exact (GPU ids mapped through the keys); filtered outputs and gradients
within relative L2 1e-4 of the fp64 oracle (fp32 atomics make the GPU's
summation order nondeterministic) and, row by row, within 1e-3 of the
row's norm plus 1e-6 of the rows' root-mean-square norm; barycentric
weights of the records the filter kernels read within 1e-6 absolute.
"""
import numpy as np
import pytest

import synth
from helpers import (assert_bary_close, assert_lattice_equal, df_term_scale, gpu_run, group_part, log, rel_l2,
                     row_errors)

pytestmark = pytest.mark.gpu

TOL = 1e-4
ROW_REL, ROW_ABS = 1e-3, 1e-6


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1907_00641_amd.binding as B

    B.lib()  # raises if the library is not built


def olat_points(olat):
    """Points with the row norms of the features the oracle lattice was
    built from: E^T E = alpha^2 I, so |x_i| / alpha = |f_i|."""
    from oracle import oracle as O

    return olat.simp.xelev / O.alpha(olat.d)


def check_array(name, got, want, msg, extra=None):
    """Whole-array relative L2 <= TOL and the per-row bound (``extra``: a
    per-row allowance for cancelling terms, added to the bound); appends
    both figures (and the worst row) to msg."""
    e = rel_l2(got, want)
    ratio, row, rerr = row_errors(got, want, ROW_REL, ROW_ABS, extra)
    msg += f" {name} {e:.2e} (worst row {row}: {rerr:.1e} of its norm, {ratio:.2f} of its bound)"
    assert e < TOL and ratio <= 1.0, msg
    return msg


def check_filter(res, O, olat, v, g, flags, bwd=True, df_is_zero=False):
    """Relative L2 error and per-row errors against the oracle.
    ``df_is_zero`` marks cases whose exact embedding gradient vanishes
    because its terms cancel (a lone point in normalised mode, where
    out = v whatever f is): there the GPU value is fp32 cancellation noise
    and is bounded in absolute terms by 1e-5 of the size |v| |g| of the
    cancelling terms."""
    norm = bool(flags & 1)
    out, st = O.forward(olat, v, norm)
    msg = check_array("out", res["out"], out, "")
    if bwd:
        dv, df = O.backward(olat, v, g, norm, st)
        if res.get("dv") is not None:
            msg = check_array("dv", res["dv"], dv, msg)
        if res.get("df") is not None:
            if df_is_zero:
                scale = np.linalg.norm(v) * np.linalg.norm(g)
                assert np.abs(df).max() < 1e-12 * scale
                e = float(np.abs(res["df"]).max() / scale)
                msg += f" |df|/(|v||g|) {e:.2e}"
                assert e < 1e-5, msg
            else:
                cancel = 1e-5 * df_term_scale(olat_points(olat), v, g, out, dv)
                msg = check_array("df", res["df"], df, msg, cancel)
    log(f"  {msg}")


# ---------------------------------------------------------------------------
# workload-shaped cases
# ---------------------------------------------------------------------------

CASES = [
    ("C1", None, False),           # 32^3, d=3, integer-grid ties, fwd only
    ("C1", (12, 12, 12), False),   # the corner checked against brute force
    ("C2", None, True),            # 64^3, d=5, C=16
    ("C2", (13, 11, 7), True),     # ragged: partial tiles everywhere
    ("C4", (40, 36, 24), True),    # d=8 recipe, reduced
    ("C5", (48, 40, 32), True),    # d=4 + intensity, C=64, reduced
]


@pytest.mark.parametrize("name,shape,bwd", CASES, ids=[f"{c[0]}-{c[1]}" for c in CASES])
@pytest.mark.parametrize("flags", [0, 1], ids=["raw", "normalized"])
def test_workload_parity(O, name, shape, bwd, flags):
    data = synth.generate(name, shape=shape)
    log(f"[parity] {name} shape={shape} flags={flags} n={data['f'].shape[0]} d={data['f'].shape[1]}")
    res = gpu_run(data["f"], data["v"], data["g"], flags, bwd=bwd)
    olat = O.lattice(data["f"])
    assert_lattice_equal(res, olat)
    assert_bary_close(res, olat)
    check_filter(res, O, olat, data["v"], data["g"], flags, bwd)


def test_headline_full_size(O):
    """128^3 voxels, d=5, C=32: the configuration the benchmark times."""
    data = synth.generate("C3")
    log(f"[parity] C3 full size n={data['f'].shape[0]}")
    res = gpu_run(data["f"], data["v"], data["g"], 0, bwd=True)
    olat = O.lattice(data["f"])
    assert_lattice_equal(res, olat)
    assert_bary_close(res, olat)
    check_filter(res, O, olat, data["v"], data["g"], 0, True)


def test_batch_full_size(O):
    """The two 160x160x96 d=8 volumes, C=16, as the benchmark times them (one
    batched build, one filter call per direction): each volume's lattice,
    output and gradients against the oracle on that volume alone."""
    vols = [synth.generate("C4", volume=b) for b in range(2)]
    n0 = vols[0]["f"].shape[0]
    starts = [0, n0, 2 * n0]
    log(f"[parity] C4 full size 2 x {n0}")
    cat = {k: np.concatenate([x[k] for x in vols]) for k in ("f", "v", "g")}
    res = gpu_run(cat["f"], cat["v"], cat["g"], 0, group_start=starts)
    total_m = 0
    for b, x in enumerate(vols):
        a, e = starts[b], starts[b + 1]
        olat = O.lattice(x["f"])
        total_m += olat.M
        assert_lattice_equal(group_part(res, b, a, e), olat)
        check_filter({k: res[k][a:e] for k in ("out", "dv", "df")}, O, olat, x["v"], x["g"], 0)
    assert res["M"] == total_m


def test_wide_channels_full_size(O):
    """192^3 voxels, d=4, C=64 as the benchmark times it: lattice and
    weights bit-exact / within 1e-6 for every point; out, dL/dv and dL/df
    compared in full (whole-array and per-row bounds)."""
    data = synth.generate("C5")
    n = data["f"].shape[0]
    log(f"[parity] C5 full size n={n}")
    res = gpu_run(data["f"], data["v"], data["g"], 0)
    olat = O.lattice(data["f"])
    assert_lattice_equal(res, olat)
    assert_bary_close(res, olat)
    check_filter(res, O, olat, data["v"], data["g"], 0, True)


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def test_empty_input():
    import torch

    import paper_1907_00641_amd as P

    log("[edge] empty")
    ft = torch.zeros((0, 3), device="cuda:0")
    lat = P.pam_lattice_build(ft)
    assert P.pam_lattice_stats(lat)[0] == 0
    v = torch.zeros((0, 4), device="cuda:0")
    out = P.pam_filter_fwd(lat, v)
    dv, df = P.pam_filter_bwd(lat, v, v)
    assert out.shape == (0, 4) and dv.shape == (0, 4) and df.shape == (0, 3)
    lat.destroy()


@pytest.mark.parametrize("d", [1, 3, 5, 8, 16])
def test_single_point(O, d):
    log(f"[edge] single point d={d}")
    f = synth.random_points(1, d, 3.0, 10 + d)
    rng = np.random.default_rng(d)
    v = rng.standard_normal((1, 5)).astype(np.float32)
    g = rng.standard_normal((1, 5)).astype(np.float32)
    for flags in (0, 1):
        res = gpu_run(f, v, g, flags)
        olat = O.lattice(f)
        assert res["M"] == d + 1
        assert_lattice_equal(res, olat)
        check_filter(res, O, olat, v, g, flags, df_is_zero=bool(flags))


@pytest.mark.parametrize("d", [2, 5])
def test_all_points_identical(O, d):
    """Maximum contention: every point splats onto the same d+1 vertices."""
    log(f"[edge] identical points d={d}")
    n = 20000
    f = np.tile(synth.random_points(1, d, 2.0, 20 + d), (n, 1))
    rng = np.random.default_rng(30 + d)
    v = rng.standard_normal((n, 8)).astype(np.float32)
    g = rng.standard_normal((n, 8)).astype(np.float32)
    res = gpu_run(f, v, g, 0)
    olat = O.lattice(f)
    assert res["M"] == d + 1
    assert_lattice_equal(res, olat)
    check_filter(res, O, olat, v, g, 0)


def test_far_apart_points_regrow(O):
    """Every point alone: M = n(d+1), beyond the first table guess, so the
    build regrows its hash table."""
    log("[edge] far apart points")
    d, n = 3, 3000
    rng = np.random.default_rng(40)
    f = rng.uniform(0, 1, size=(n, d))
    f[:, 0] += 30.0 * np.arange(n)
    f = f.astype(np.float32)
    v = rng.standard_normal((n, 4)).astype(np.float32)
    g = rng.standard_normal((n, 4)).astype(np.float32)
    res = gpu_run(f, v, g, 0)
    olat = O.lattice(f)
    assert res["M"] == n * (d + 1)
    assert_lattice_equal(res, olat)
    check_filter(res, O, olat, v, g, 0)


def test_capacity_hint_regrow_and_refusal(O):
    import torch

    import paper_1907_00641_amd as P

    log("[edge] capacity hint")
    data = synth.generate("C2", shape=(20, 18, 16))
    ft = torch.from_numpy(data["f"]).cuda()
    olat = O.lattice(data["f"])
    lat = P.pam_lattice_build(ft)
    P.pam_lattice_set_capacity(lat, 64, allow_regrow=True)
    P.pam_lattice_build(ft, lat=lat)
    M, cap = P.pam_lattice_stats(lat)
    assert M == olat.M and cap >= 2 * M
    keys, vert, bary, nbr = P.pam_lattice_export(lat)
    assert_lattice_equal({"M": M, "keys": keys, "vert": vert, "nbr": nbr}, olat)
    P.pam_lattice_set_capacity(lat, 64, allow_regrow=False)
    with pytest.raises(P.PamError) as ei:
        P.pam_lattice_build(ft, lat=lat)
    assert ei.value.status == 3  # PAM_ERR_CAPACITY
    P.pam_lattice_set_capacity(lat, 0, allow_regrow=True)
    P.pam_lattice_build(ft, lat=lat)
    assert P.pam_lattice_stats(lat)[0] == olat.M
    lat.destroy()


def test_large_table_small_lattice(O):
    """A 2^21-slot table under a lattice of a few thousand vertices: the
    compaction of tables from 2^20 slots (16 slots per thread, most blocks
    without a key) must still give dense ids, and the filter must match."""
    import torch

    import paper_1907_00641_amd as P

    log("[edge] large table, small lattice")
    data = synth.generate("C2", shape=(20, 18, 16))
    f, v, g = data["f"], data["v"][:, :8].copy(), data["g"][:, :8].copy()
    olat = O.lattice(f)
    ft = torch.from_numpy(f).cuda()
    lat = P.pam_lattice_build(ft)
    P.pam_lattice_set_capacity(lat, 1 << 21, allow_regrow=False)
    P.pam_lattice_build(ft, lat=lat)
    M, cap = P.pam_lattice_stats(lat)
    assert cap == 1 << 21 and M == olat.M
    keys, vert, bary, nbr = P.pam_lattice_export(lat)
    assert_lattice_equal({"M": M, "keys": keys, "vert": vert, "nbr": nbr}, olat)
    vt, gt = torch.from_numpy(v).cuda(), torch.from_numpy(g).cuda()
    out = P.pam_filter_fwd(lat, vt)
    dv, df = P.pam_filter_bwd(lat, vt, gt)
    res = {"out": out.cpu().numpy(), "dv": dv.cpu().numpy(), "df": df.cpu().numpy()}
    lat.destroy()
    check_filter(res, O, olat, v, g, 0)


@pytest.mark.parametrize("bad", ["huge", "nan", "inf"])
def test_key_range_errors(bad):
    import torch

    import paper_1907_00641_amd as P

    log(f"[edge] key range {bad}")
    f = synth.random_points(500, 3, 4.0, 50)
    f[123, 1] = {"huge": 1e9, "nan": np.nan, "inf": np.inf}[bad]
    ft = torch.from_numpy(f).cuda()
    with pytest.raises(P.PamError) as ei:
        P.pam_lattice_build(ft)
    assert ei.value.status == 4  # PAM_ERR_KEY_RANGE


def test_state_errors():
    import torch

    import paper_1907_00641_amd as P

    log("[edge] state errors")
    f = torch.from_numpy(synth.random_points(300, 3, 4.0, 60)).cuda()
    v = torch.randn(300, 4, device="cuda:0")
    lat = P.pam_lattice_build(f)
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_bwd(lat, v, v)
    assert ei.value.status == 5
    P.pam_filter_fwd(lat, v)
    v8 = torch.randn(300, 8, device="cuda:0")
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_bwd(lat, v8, v8)
    assert ei.value.status == 5
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_bwd(lat, v, v, flags=1)
    assert ei.value.status == 5
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_fwd(lat, v, flags=4)
    assert ei.value.status == 1
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_fwd(lat, v, out=v)
    assert ei.value.status == 1
    P.pam_lattice_build(f, lat=lat)  # rebuild invalidates the forward state
    with pytest.raises(P.PamError) as ei:
        P.pam_filter_bwd(lat, v, v)
    assert ei.value.status == 5
    lat.destroy()


@pytest.mark.parametrize("which", ["grad_val_only", "grad_feat_only"])
@pytest.mark.parametrize("flags", [0, 1])
def test_optional_gradients(O, which, flags):
    log(f"[edge] {which} flags={flags}")
    data = synth.generate("C2", shape=(17, 15, 9))
    gv, gf = (True, None) if which == "grad_val_only" else (None, True)
    res = gpu_run(data["f"], data["v"], data["g"], flags, grad_val=gv, grad_feat=gf)
    assert (res["dv"] is None) == (gv is None) and (res["df"] is None) == (gf is None)
    olat = O.lattice(data["f"])
    check_filter(res, O, olat, data["v"], data["g"], flags)


@pytest.mark.parametrize("C", [1, 7, 33, 1024])
def test_channel_counts(O, C):
    log(f"[edge] C={C}")
    f = synth.random_points(700 if C < 1024 else 150, 4, 4.0, 70 + C)
    rng = np.random.default_rng(C)
    v = rng.standard_normal((f.shape[0], C)).astype(np.float32)
    g = rng.standard_normal((f.shape[0], C)).astype(np.float32)
    olat = O.lattice(f)
    for flags in (0, 1):
        res = gpu_run(f, v, g, flags)
        check_filter(res, O, olat, v, g, flags)


@pytest.mark.parametrize("d,C", [(3, 4), (3, 8), (5, 12), (5, 16), (6, 8), (7, 12), (8, 4), (8, 16), (8, 20)])
def test_narrow_channel_groups(O, d, C):
    """Rows of at most 8 or 16 channels take 2- or 4-lane groups in the
    splat and both slices (d <= 8); d >= 6 also takes 256-point tiles, where
    the splat copies the tile's rows of x to LDS (C = 4, 8, 12, 16: lanes
    past C read zeros).  Raw and normalised (the weight column widens the
    lattice row), over several tiles with a ragged last one."""
    log(f"[edge] narrow groups d={d} C={C}")
    f = synth.random_points(1700, d, 3.0, 300 + 10 * d + C)
    rng = np.random.default_rng(900 + C)
    v = rng.standard_normal((f.shape[0], C)).astype(np.float32)
    g = rng.standard_normal((f.shape[0], C)).astype(np.float32)
    olat = O.lattice(f)
    for flags in (0, 1):
        res = gpu_run(f, v, g, flags)
        assert_lattice_equal(res, olat)
        check_filter(res, O, olat, v, g, flags)


@pytest.mark.parametrize("d", [1, 2, 7, 12, 16])
def test_dimensions(O, d):
    log(f"[edge] d={d}")
    f = synth.random_points(1500, d, 3.0, 80 + d)
    rng = np.random.default_rng(90 + d)
    v = rng.standard_normal((1500, 6)).astype(np.float32)
    g = rng.standard_normal((1500, 6)).astype(np.float32)
    res = gpu_run(f, v, g, 0)
    olat = O.lattice(f)
    assert_lattice_equal(res, olat)
    assert_bary_close(res, olat)
    check_filter(res, O, olat, v, g, 0)


def test_rebuild_reuses_handle_across_shapes(O):
    import torch

    import paper_1907_00641_amd as P

    log("[edge] handle reuse")
    lat = None
    for k, (name, shape) in enumerate([("C2", (24, 20, 16)), ("C1", (16, 16, 8)), ("C4", (20, 16, 12)),
                                       ("C2", (24, 20, 16))]):
        data = synth.generate(name, shape=shape)
        ft = torch.from_numpy(data["f"]).cuda()
        vt = torch.from_numpy(data["v"]).cuda()
        gt = torch.from_numpy(data["g"]).cuda()
        lat = P.pam_lattice_build(ft, lat=lat)
        out = P.pam_filter_fwd(lat, vt)
        dv, df = P.pam_filter_bwd(lat, vt, gt)
        keys, vert, bary, nbr = P.pam_lattice_export(lat)
        M, _ = P.pam_lattice_stats(lat)
        olat = O.lattice(data["f"])
        assert_lattice_equal({"M": M, "keys": keys, "vert": vert, "nbr": nbr}, olat)
        check_filter({"out": out.cpu().numpy(), "dv": dv.cpu().numpy(), "df": df.cpu().numpy()},
                     O, olat, data["v"], data["g"], 0)
    lat.destroy()


def test_rebuild_outside_fixed_key_layout(O):
    """Rebuilds of a handle pack keys with a fixed layout (d = 5: 12 bits
    per stored quotient, centred on zero) without measuring the range;
    features whose quotients leave it (here every coordinate shifted by
    2000, quotients of about 3600) make the insert flag the build, which is
    then redone with the layout taken from the measured range.  Small, then
    shifted, then small features again on one handle: each build matches
    the oracle's lattice bit for bit and its filter."""
    import torch

    import paper_1907_00641_amd as P

    log("[edge] rebuild outside the fixed key layout")
    d, n = 5, 3000
    rng = np.random.default_rng(41)
    small = rng.uniform(0.0, 4.0, size=(n, d)).astype(np.float32)
    shifted = (small + np.float32(2000.0)).astype(np.float32)
    v = rng.standard_normal((n, 8)).astype(np.float32)
    g = rng.standard_normal((n, 8)).astype(np.float32)
    vt, gt = torch.from_numpy(v).cuda(), torch.from_numpy(g).cuda()
    lat, fast_seen, miss_seen = None, 0, 0
    for f in (small, small, shifted, small, shifted, small):
        ft = torch.from_numpy(f).cuda()
        cap0 = None
        if lat is not None:
            cap0 = P.pam_lattice_stats(lat)[1]
            P.pam_timing_enable(lat, True)
        lat = P.pam_lattice_build(ft, lat=lat)
        if cap0 is not None and P.pam_lattice_stats(lat)[1] == cap0:
            # same table capacity as the build before, which left the table
            # empty: small features take the fast insert alone, shifted ones
            # a fast attempt and then the range pass
            launches = {name: c for name, (c, _) in P.pam_timing_read(lat).items()}
            want = (0, 1) if f is small else (1, 2)
            assert (launches.get("range", 0), launches.get("insert", 0)) == want, launches
            fast_seen += f is small
            miss_seen += f is shifted
        if cap0 is not None:
            P.pam_timing_enable(lat, False)
        out = P.pam_filter_fwd(lat, vt)
        dv, df = P.pam_filter_bwd(lat, vt, gt)
        keys, vert, bary, nbr = P.pam_lattice_export(lat)
        M, _ = P.pam_lattice_stats(lat)
        olat = O.lattice(f)
        assert_lattice_equal({"M": M, "keys": keys, "vert": vert, "nbr": nbr}, olat)
        assert_bary_close({"bary": bary}, olat)
        check_filter({"out": out.cpu().numpy(), "dv": dv.cpu().numpy(), "df": df.cpu().numpy()},
                     O, olat, v, g, 0)
    lat.destroy()
    assert fast_seen >= 1 and miss_seen >= 1, (fast_seen, miss_seen)


def test_call_sequences_reuse_cleared_lattices(O):
    """The build clears the splat targets of the next forward and backward
    calls for the last row stride used, and those calls then skip their own
    clearing.  Sequences that break that assumption (a larger lattice after
    a rebuild, more channels, normalised mode, repeated calls, asymmetric
    calls in between) must still match the oracle at every call."""
    import torch

    import paper_1907_00641_amd as P

    small = synth.generate("C2", shape=(14, 12, 10))
    large = synth.generate("C2", shape=(26, 22, 18))
    rng = np.random.default_rng(77)

    def vals(n, c):
        return rng.standard_normal((n, c)).astype(np.float32)

    lat = None
    olats = {}
    # (features, C, flags, forward calls, backward calls after the last forward)
    seq = [(small, 8, 0, 1, 1), (large, 8, 0, 1, 1), (large, 16, 0, 1, 1), (large, 16, 0, 2, 2),
           (small, 16, 1, 1, 1), (small, 16, 0, 1, 1), (large, 4, 1, 1, 2), (large, 4, 1, 1, 1)]
    for step, (data, C, flags, nf, nb) in enumerate(seq):
        f = data["f"]
        key = id(data)
        if key not in olats:
            olats[key] = O.lattice(f)
        olat = olats[key]
        ft = torch.from_numpy(f).cuda()
        lat = P.pam_lattice_build(ft, lat=lat)
        for _ in range(nf):
            v = vals(f.shape[0], C)
            vt = torch.from_numpy(v).cuda()
            out = P.pam_filter_fwd(lat, vt, flags)
        for _ in range(nb):
            g = vals(f.shape[0], C)
            gt = torch.from_numpy(g).cuda()
            dv, df = P.pam_filter_bwd(lat, vt, gt, flags)
            log(f"[sequence] step {step} n={f.shape[0]} C={C} flags={flags}")
            check_filter({"out": out.cpu().numpy(), "dv": dv.cpu().numpy(), "df": df.cpu().numpy()},
                         O, olat, v, g, flags)
        if step == 3:  # an asymmetric pair on the same lattice between symmetric calls
            nk = f.shape[0] // 2
            va = vals(nk, C)
            oa = P.pam_filter_fwd_asym(lat, nk, torch.from_numpy(va).cuda())
            want = O.forward_asym(olat, nk, va)[0]
            check_array("asymmetric out", oa.cpu().numpy(), want, "")
    lat.destroy()


def test_side_streams_and_concurrent_handles(O):
    """Two handles driven from two side streams (default priority), their
    calls interleaved so that the streams overlap: build, forward and
    backward run on the stream passed in, and each handle's results match
    the oracle on its own points (different d and C on the two)."""
    import torch

    import paper_1907_00641_amd as P

    cases = [synth.generate("C2", shape=(22, 18, 14)), synth.generate("C4", shape=(18, 16, 12))]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    main = torch.cuda.current_stream()
    ft, vt, gt = [], [], []
    for data in cases:
        ft.append(torch.from_numpy(data["f"]).cuda())
        vt.append(torch.from_numpy(data["v"]).cuda())
        gt.append(torch.from_numpy(data["g"]).cuda())
    for st in streams:
        st.wait_stream(main)  # the inputs were written on the default stream
    lats, outs, grads = [None, None], [None, None], [None, None]
    for k in range(2):
        with torch.cuda.stream(streams[k]):
            lats[k] = P.pam_lattice_build(ft[k], stream=streams[k])
    for k in range(2):
        with torch.cuda.stream(streams[k]):
            outs[k] = P.pam_filter_fwd(lats[k], vt[k], stream=streams[k])
    for k in range(2):
        with torch.cuda.stream(streams[k]):
            grads[k] = P.pam_filter_bwd(lats[k], vt[k], gt[k], stream=streams[k])
    for st in streams:
        st.synchronize()
    for k, data in enumerate(cases):
        olat = O.lattice(data["f"])
        log(f"[streams] handle {k} n={data['f'].shape[0]} d={data['f'].shape[1]} C={data['v'].shape[1]}")
        check_filter({"out": outs[k].cpu().numpy(), "dv": grads[k][0].cpu().numpy(), "df": grads[k][1].cpu().numpy()},
                     O, olat, data["v"], data["g"], 0)
        lats[k].destroy()


def test_repeated_builds_are_deterministic():
    """The vertex set and the per-point vertex keys do not depend on the
    order in which concurrent insertions land."""
    import torch

    import paper_1907_00641_amd as P
    from helpers import canonical_perm

    log("[stress] repeated builds")
    data = synth.generate("C2")
    ft = torch.from_numpy(data["f"]).cuda()
    lat = P.pam_lattice_build(ft)
    ref = None
    for _ in range(10):
        P.pam_lattice_build(ft, lat=lat)
        keys, vert, _, _ = P.pam_lattice_export(lat)
        order, perm = canonical_perm(keys)
        cur = (keys[order].tobytes(), perm[vert].tobytes())
        if ref is None:
            ref = cur
        assert cur == ref
    lat.destroy()


@pytest.mark.parametrize("flags", [0, 1])
def test_tile_overflow_fallback(O, flags):
    """d=8 isolated points: each tile of 512 points has 4608 distinct
    vertices, more than the build's per-tile table holds, so the splat
    kernels take their direct-atomic path for those tiles."""
    log(f"[edge] tile overflow flags={flags}")
    d, n = 8, 1100
    rng = np.random.default_rng(120)
    f = rng.uniform(0, 1, size=(n, d))
    f[:, 0] += 20.0 * np.arange(n)
    f = f.astype(np.float32)
    v = rng.standard_normal((n, 12)).astype(np.float32)
    g = rng.standard_normal((n, 12)).astype(np.float32)
    res = gpu_run(f, v, g, flags)
    olat = O.lattice(f)
    assert res["M"] == n * (d + 1)
    assert_lattice_equal(res, olat)
    # isolated points: in normalised mode out = v, so dL/df is exactly 0
    check_filter(res, O, olat, v, g, flags, df_is_zero=bool(flags))


def test_large_lattice_unfused_blur(O):
    """A lattice too large for the fused two-direction blur (M * ld * 4 bytes
    above 32 MiB: 2200 isolated points in d=3 give 8800 vertices of 1024
    channels) takes one launch per direction; same bar as everywhere."""
    log("[edge] unfused blur")
    d, n, C = 3, 2200, 1024
    rng = np.random.default_rng(130)
    f = rng.uniform(0, 1, size=(n, d))
    f[:, 0] += 20.0 * np.arange(n)
    f = f.astype(np.float32)
    v = rng.standard_normal((n, C)).astype(np.float32)
    g = rng.standard_normal((n, C)).astype(np.float32)
    res = gpu_run(f, v, g, 0)
    olat = O.lattice(f)
    assert res["M"] * C * 4 > 32 << 20
    check_filter(res, O, olat, v, g, 0)



# ---------------------------------------------------------------------------
# batched builds: independent point groups in one launch sequence
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("flags", [0, 1], ids=["raw", "normalized"])
def test_groups_match_independent_lattices(O, flags):
    """Both volumes of the d=8 batch recipe (reduced), built together as two
    groups: each group's lattice, outputs and gradients equal those of the
    volume filtered alone."""
    shape = (20, 16, 12)
    vols = [synth.generate("C4", volume=b, shape=shape) for b in range(2)]
    log(f"[groups] C4 x2 shape={shape} flags={flags}")
    f = np.concatenate([x["f"] for x in vols])
    v = np.concatenate([x["v"] for x in vols])
    g = np.concatenate([x["g"] for x in vols])
    n0 = vols[0]["f"].shape[0]
    starts = [0, n0, f.shape[0]]
    res = gpu_run(f, v, g, flags, group_start=starts)
    total_m = 0
    for b, x in enumerate(vols):
        a, e = starts[b], starts[b + 1]
        olat = O.lattice(x["f"])
        total_m += olat.M
        assert_lattice_equal(group_part(res, b, a, e), olat)
        sub = {k: res[k][a:e] for k in ("out", "dv", "df")}
        check_filter(sub, O, olat, x["v"], x["g"], flags)
    assert res["M"] == total_m


def test_groups_identical_features_do_not_interact(O):
    """Three groups, the middle one empty, the outer two with the same
    features and different values: each outer group filters alone."""
    log("[groups] identical features, empty group")
    f1 = synth.random_points(900, 4, 3.0, 140)
    rng = np.random.default_rng(141)
    v = rng.standard_normal((1800, 9)).astype(np.float32)
    g = rng.standard_normal((1800, 9)).astype(np.float32)
    f = np.concatenate([f1, f1])
    starts = [0, 900, 900, 1800]
    res = gpu_run(f, v, g, 0, group_start=starts)
    olat = O.lattice(f1)
    assert res["M"] == 2 * olat.M
    for grp, (a, e) in ((0, (0, 900)), (2, (900, 1800))):
        assert_lattice_equal(group_part(res, grp, a, e), olat)
        check_filter({k: res[k][a:e] for k in ("out", "dv", "df")}, O, olat, v[a:e], g[a:e], 0)


def augmented_case(d, C, n_or_shape, seed):
    if isinstance(n_or_shape, str):  # "C3:48x40x32": that workload's recipe at a reduced volume
        name, dims = n_or_shape.split(":")
        data = synth.generate(name, shape=tuple(int(x) for x in dims.split("x")))
        return data["f"], data["v"], data["g"]
    if isinstance(n_or_shape, tuple):
        data = synth.generate("C2", shape=n_or_shape)
        rng = np.random.default_rng(seed)
        f = data["f"]
        v = rng.standard_normal((f.shape[0], C)).astype(np.float32)
        g = rng.standard_normal((f.shape[0], C)).astype(np.float32)
        return f, v, g
    f = synth.random_points(n_or_shape, d, 4.0, seed)
    rng = np.random.default_rng(seed + 1)
    v = rng.standard_normal((n_or_shape, C)).astype(np.float32)
    g = rng.standard_normal((n_or_shape, C)).astype(np.float32)
    return f, v, g


@pytest.mark.parametrize("d,C,size", [(3, 8, 3000), (5, 32, (20, 18, 14)), (5, 7, (17, 13, 11)), (2, 40, 2500),
                                      (8, 4, 1500), (5, 32, "C3:48x40x32")],
                         ids=["d3c8", "d5c32", "d5c7", "d2c40", "d8c4", "c3recipe"])
def test_augmented_embedding_gradient(O, d, C, size):
    """PAM_EGRAD_AUGMENTED: the embedding gradient from filters of f (x) v
    and f (x) g (several 32-channel chunks, ragged chunks, scalar-lane
    rows, and the 128^3 workload's recipe on a 48x40x32 volume: 120 full
    512-point tiles like the benchmarked ones) against the oracle's
    estimator; the value gradient is unchanged."""
    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    f, v, g = augmented_case(d, C, size, 1600 + d + C)
    log(f"[augmented] d={d} C={C} n={f.shape[0]}")
    dev = torch.device("cuda:0")
    ft, vt, gt = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (f, v, g))
    lat = P.pam_lattice_build(ft)
    P.pam_filter_fwd(lat, vt, 0)
    dv, df = P.pam_filter_bwd(lat, vt, gt, B.PAM_EGRAD_AUGMENTED)
    _, df8 = P.pam_filter_bwd(lat, vt, gt, 0, grad_val=False)
    torch.cuda.synchronize()
    dv, df, df8 = dv.cpu().numpy(), df.cpu().numpy(), df8.cpu().numpy()
    lat.destroy()
    olat = O.lattice(f)
    out, st = O.forward(olat, v, False)
    odv, odf8 = O.backward(olat, v, g, False, st)
    odf = O.backward_augmented(olat, f, v, g)
    cancel = 1e-5 * df_term_scale(f, v, g, out, odv)
    msg = check_array("augmented df", df, odf, "", cancel)
    msg = check_array("dv", dv, odv, msg)
    log("  " + check_array("eq. 8 df", df8, odf8, msg, cancel))


@pytest.mark.parametrize("d,C,scale", [(12, 4, 1.0), (16, 6, 0.5)], ids=["d12c4", "d16c6"])
def test_augmented_high_dimensions(O, d, C, scale):
    """PAM_EGRAD_AUGMENTED above d = 8, where a tile's d+1 values per
    contribution do not all fit the augmented slice's LDS slots and are
    taken in chunks (7 of 13 values per chunk at d=12, 5 of 17 at d=16);
    C = 6 runs scalar-lane rows (32-lane groups, whole-group sums) and C = 4
    two-lane groups (reduce-scatter).  Clustered points (the whole lattice
    under 4096 vertices) keep every tile within the build's per-tile table."""
    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    n = 900
    log(f"[augmented] d={d} C={C} n={n}")
    f = synth.random_points(n, d, scale, 1700 + d)
    rng = np.random.default_rng(1701 + d)
    v = rng.standard_normal((n, C)).astype(np.float32)
    g = rng.standard_normal((n, C)).astype(np.float32)
    olat = O.lattice(f)
    assert olat.M <= 4096
    dev = torch.device("cuda:0")
    ft, vt, gt = (torch.from_numpy(a).to(dev) for a in (f, v, g))
    lat = P.pam_lattice_build(ft)
    P.pam_filter_fwd(lat, vt, 0)
    dv, df = P.pam_filter_bwd(lat, vt, gt, B.PAM_EGRAD_AUGMENTED)
    torch.cuda.synchronize()
    dv, df = dv.cpu().numpy(), df.cpu().numpy()
    lat.destroy()
    out, st = O.forward(olat, v, False)
    odv, _ = O.backward(olat, v, g, False, st)
    odf = O.backward_augmented(olat, f, v, g)
    cancel = 1e-5 * df_term_scale(f, v, g, out, odv)
    msg = check_array("augmented df", df, odf, "", cancel)
    log("  " + check_array("dv", dv, odv, msg))


def test_augmented_overflow_tiles(O):
    """PAM_EGRAD_AUGMENTED on tiles whose vertices overflow the build's
    per-tile table: d=8 pairs of points 1.5 apart, the pairs on a grid of
    spacing 20 (|f| stays small: the estimator's f (x) v - f Wv cancels in
    proportion to |f|), so that the points of a pair interact (a non-zero
    gradient) while 256 points of full pairs have more distinct vertices
    than the table's 2048 slots (checked on the oracle's lattice below; the
    pairs share no vertex, and a pair split over two tiles gives each 9).
    The full tiles take the per-point paths of the augmented splat and
    slice, the last (76 points) the tiled ones; same bar as elsewhere."""
    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    d, n, C = 8, 1100, 12
    log(f"[augmented] overflow tiles d={d} C={C} n={n}")
    rng = np.random.default_rng(122)
    npair = n // 2
    digits = (np.arange(npair)[:, None] // 3 ** np.arange(d)[None, :]) % 3
    base = 20.0 * (digits - 1) + rng.uniform(0, 1, size=(npair, d))
    dirs = rng.standard_normal((npair, d))
    dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
    f = np.empty((n, d))
    f[0::2] = base
    f[1::2] = base + 1.5 * dirs
    f = f.astype(np.float32)
    v = rng.standard_normal((n, C)).astype(np.float32)
    g = rng.standard_normal((n, C)).astype(np.float32)
    olat = O.lattice(f)
    per_pair = np.sort([len(set(olat.vert[2 * j]) | set(olat.vert[2 * j + 1])) for j in range(npair)])
    assert per_pair.sum() == olat.M  # no vertex shared between pairs
    assert per_pair[:128].sum() > 2048  # any 128 full pairs overflow the table
    dev = torch.device("cuda:0")
    ft, vt, gt = (torch.from_numpy(a).to(dev) for a in (f, v, g))
    lat = P.pam_lattice_build(ft)
    P.pam_filter_fwd(lat, vt, 0)
    dv, df = P.pam_filter_bwd(lat, vt, gt, B.PAM_EGRAD_AUGMENTED)
    torch.cuda.synchronize()
    dv, df = dv.cpu().numpy(), df.cpu().numpy()
    lat.destroy()
    out, st = O.forward(olat, v, False)
    odv, _ = O.backward(olat, v, g, False, st)
    odf = O.backward_augmented(olat, f, v, g)
    assert np.linalg.norm(odf) > 0.1 * np.linalg.norm(odv)  # the pairs interact
    cancel = 1e-5 * df_term_scale(f, v, g, out, odv)
    msg = check_array("augmented df", df, odf, "", cancel)
    log("  " + check_array("dv", dv, odv, msg))


def test_augmented_flag_errors(O):
    """PAM_EGRAD_AUGMENTED needs raw mode and belongs to the backward call."""
    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    f, v, g = augmented_case(3, 4, 500, 1700)
    dev = torch.device("cuda:0")
    ft, vt, gt = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (f, v, g))
    lat = P.pam_lattice_build(ft)
    L = B.lib()
    out = torch.empty_like(vt)
    assert L.pam_filter_fwd(lat.handle, vt.data_ptr(), 4, B.PAM_EGRAD_AUGMENTED, out.data_ptr(),
                            None) == B.PAM_ERR_INVALID_ARGUMENT
    P.pam_filter_fwd(lat, vt, B.PAM_NORMALIZE, out=out)
    dfb = torch.empty_like(ft)
    rc = L.pam_filter_bwd(lat.handle, vt.data_ptr(), gt.data_ptr(), 4, B.PAM_NORMALIZE | B.PAM_EGRAD_AUGMENTED,
                          None, dfb.data_ptr(), None)
    assert rc == B.PAM_ERR_INVALID_ARGUMENT
    # raw forward state: the augmented flag is accepted with the raw forward
    P.pam_filter_fwd(lat, vt, 0, out=out)
    rc = L.pam_filter_bwd(lat.handle, vt.data_ptr(), gt.data_ptr(), 4, B.PAM_EGRAD_AUGMENTED, None,
                          dfb.data_ptr(), None)
    assert rc == B.PAM_OK
    torch.cuda.synchronize()
    lat.destroy()


def asym_points(d, nk, nq, seed, C):
    rng = np.random.default_rng(seed)
    k = synth.random_points(nk, d, 4.0, seed)
    q = (synth.random_points(nq, d, 4.0, seed + 1) + np.float32(0.41)).astype(np.float32)
    v = rng.standard_normal((nk, C)).astype(np.float32)
    g = rng.standard_normal((nq, C)).astype(np.float32)
    return k, q, v, g


def gpu_asym(k, q, v, g, grad_val=True, grad_feat=True):
    import torch

    import paper_1907_00641_amd as P

    dev = torch.device("cuda:0")
    nk = k.shape[0]
    ft = torch.from_numpy(np.ascontiguousarray(np.concatenate([k, q]))).to(dev)
    vt = torch.from_numpy(np.ascontiguousarray(v)).to(dev)
    gt = torch.from_numpy(np.ascontiguousarray(g)).to(dev)
    lat = P.pam_lattice_build(ft)
    out = P.pam_filter_fwd_asym(lat, nk, vt)
    dv, df = P.pam_filter_bwd_asym(lat, nk, vt, gt, grad_val=grad_val, grad_feat=grad_feat)
    torch.cuda.synchronize()
    res = {"out": out.cpu().numpy(), "dv": None if dv is None else dv.cpu().numpy(),
           "df": None if df is None else df.cpu().numpy(), "M": P.pam_lattice_stats(lat)[0]}
    lat.destroy()
    return res


@pytest.mark.parametrize("d,nk,nq,C", [(3, 2500, 1800, 8), (5, 3000, 2000, 32), (5, 1500, 2600, 7), (2, 2000, 900, 40),
                                       (8, 1200, 1100, 4)],
                         ids=["d3c8", "d5c32", "d5c7", "d2c40", "d8c4"])
def test_asym_matches_oracle(O, d, nk, nq, C):
    """Asymmetric filter (values at the keys, read at the queries) through
    the C ABI against the oracle: out, dL/dv (keys) and dL/df (keys and
    queries)."""
    k, q, v, g = asym_points(d, nk, nq, 2100 + d + C, C)
    log(f"[asym] d={d} nk={nk} nq={nq} C={C}")
    res = gpu_asym(k, q, v, g)
    lat = O.lattice(np.concatenate([k, q]))
    assert res["M"] == lat.M
    out, st = O.forward_asym(lat, nk, v)
    dv, df = O.backward_asym(lat, nk, v, g, st)
    msg = check_array("out", res["out"], out, "")
    msg = check_array("dv", res["dv"], dv, msg)
    log("  " + check_array("df", res["df"], df, msg))


def test_asym_5d_volume_queries_shifted(O):
    """The d=5 volume recipe at reduced size as keys, the same voxels moved
    by a quarter voxel as queries (the tiles mix keys and queries)."""
    data = synth.generate("C2", shape=(18, 16, 12))
    k = data["f"]
    q = k.copy()
    q[:, :3] += np.float32(0.25 / 8.0)
    C = 16
    rng = np.random.default_rng(2200)
    v = rng.standard_normal((k.shape[0], C)).astype(np.float32)
    g = rng.standard_normal((q.shape[0], C)).astype(np.float32)
    res = gpu_asym(k, q, v, g)
    lat = O.lattice(np.concatenate([k, q]))
    out, st = O.forward_asym(lat, k.shape[0], v)
    dv, df = O.backward_asym(lat, k.shape[0], v, g, st)
    msg = check_array("out", res["out"], out, "")
    msg = check_array("dv", res["dv"], dv, msg)
    log("  " + check_array("df", res["df"], df, msg))


def test_asym_degenerate_splits(O):
    """No keys: the queries read 0 and both gradients vanish.  No queries:
    an empty output and vanishing gradients.  Only grad_val requested."""
    import torch

    import paper_1907_00641_amd as P

    k, q, v, g = asym_points(3, 800, 600, 2300, 4)
    dev = torch.device("cuda:0")
    # no keys
    ft = torch.from_numpy(q).to(dev)
    lat = P.pam_lattice_build(ft)
    v0 = torch.zeros((0, 4), device=dev)
    out = P.pam_filter_fwd_asym(lat, 0, v0)
    _, df = P.pam_filter_bwd_asym(lat, 0, v0, torch.from_numpy(g).to(dev), grad_val=False)
    torch.cuda.synchronize()
    assert out.shape == (600, 4) and float(out.abs().max()) == 0.0
    assert float(df.abs().max()) == 0.0
    lat.destroy()
    # no queries
    ft = torch.from_numpy(k).to(dev)
    lat = P.pam_lattice_build(ft)
    vt = torch.from_numpy(v).to(dev)
    out = P.pam_filter_fwd_asym(lat, 800, vt)
    dv, df = P.pam_filter_bwd_asym(lat, 800, vt, torch.zeros((0, 4), device=dev))
    torch.cuda.synchronize()
    assert out.shape == (0, 4)
    assert float(dv.abs().max()) == 0.0 and float(df.abs().max()) == 0.0
    lat.destroy()
    # value gradient only
    res = gpu_asym(k, q, v, g, grad_feat=False)
    lat_o = O.lattice(np.concatenate([k, q]))
    _, st = O.forward_asym(lat_o, 800, v)
    dv_o, _ = O.backward_asym(lat_o, 800, v, g, st)
    assert res["df"] is None
    check_array("dv", res["dv"], dv_o, "")


def test_asym_errors(O):
    import torch

    import paper_1907_00641_amd as P
    from paper_1907_00641_amd import binding as B

    k, q, v, g = asym_points(3, 300, 200, 2400, 4)
    dev = torch.device("cuda:0")
    ft = torch.from_numpy(np.concatenate([k, q])).to(dev)
    vt, gt = torch.from_numpy(v).to(dev), torch.from_numpy(g).to(dev)
    lat = P.pam_lattice_build(ft)
    L = B.lib()
    out = torch.empty((200, 4), device=dev)
    dfb = torch.empty_like(ft)
    assert L.pam_filter_fwd_asym(lat.handle, 300, vt.data_ptr(), 4, B.PAM_NORMALIZE, out.data_ptr(),
                                 None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_filter_fwd_asym(lat.handle, 501, vt.data_ptr(), 4, 0, out.data_ptr(),
                                 None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_filter_fwd_asym(lat.handle, -1, vt.data_ptr(), 4, 0, out.data_ptr(),
                                 None) == B.PAM_ERR_INVALID_ARGUMENT
    # backward needs the matching forward
    assert L.pam_filter_bwd_asym(lat.handle, 300, vt.data_ptr(), gt.data_ptr(), 4, 0, None, dfb.data_ptr(),
                                 None) == B.PAM_ERR_STATE
    P.pam_filter_fwd_asym(lat, 300, vt, out=out)
    assert L.pam_filter_bwd_asym(lat.handle, 299, vt.data_ptr(), gt.data_ptr(), 4, 0, None, dfb.data_ptr(),
                                 None) == B.PAM_ERR_STATE
    assert L.pam_filter_bwd_asym(lat.handle, 300, vt.data_ptr(), gt.data_ptr(), 4, B.PAM_EGRAD_AUGMENTED, None,
                                 dfb.data_ptr(), None) == B.PAM_ERR_INVALID_ARGUMENT
    assert L.pam_filter_bwd(lat.handle, vt.data_ptr(), gt.data_ptr(), 4, 0, None, dfb.data_ptr(),
                            None) == B.PAM_ERR_STATE
    torch.cuda.synchronize()
    lat.destroy()


def test_probe_copy_rows():
    """The measurement utility copies rows exactly in each of its four
    modes (read and/or write positions permuted), on a ragged row count."""
    import torch

    import paper_1907_00641_amd as P

    dev = torch.device("cuda:0")
    gen = torch.Generator().manual_seed(5)
    n, c = 1000, 12
    x = torch.randn(n, c, generator=gen).to(dev)
    perm = torch.randperm(n, generator=gen).to(torch.int32).to(dev)
    pl = perm.long()
    for mode in range(4):
        y = torch.full_like(x, float("nan"))
        P.pam_probe_copy_rows(x, y, perm, mode)
        torch.cuda.synchronize()
        want = torch.empty_like(x)
        src = x[pl] if mode & 1 else x
        if mode & 2:
            want[pl] = src
        else:
            want.copy_(src)
        assert torch.equal(y, want), f"mode {mode}"
    with pytest.raises(P.PamError):
        P.pam_probe_copy_rows(x[:, :6].contiguous(), torch.empty(n, 6, device=dev), perm, 0)


@pytest.mark.parametrize("case", ["C2", "asym", "overflow"])
def test_fused_eq8_term(O, case, monkeypatch):
    """PAM_FUSE_EQ8=1: the backward splat forms eq. 8's slice-side term
    (raw mode, C <= 32) and the backward slice reads it instead of g; same
    bar as the default path, on a volume, on the asymmetric filter (the keys
    have no row of g) and on tiles that take the direct-atomic path."""
    monkeypatch.setenv("PAM_FUSE_EQ8", "1")
    log(f"[fused eq. 8] {case}")
    if case == "C2":
        data = synth.generate("C2", shape=(26, 22, 18))
        res = gpu_run(data["f"], data["v"], data["g"], 0)
        olat = O.lattice(data["f"])
        check_filter(res, O, olat, data["v"], data["g"], 0)
    elif case == "asym":
        k, q, v, g = asym_points(5, 3000, 2000, 2500, 32)
        res = gpu_asym(k, q, v, g)
        lat = O.lattice(np.concatenate([k, q]))
        out, st = O.forward_asym(lat, 3000, v)
        dv, df = O.backward_asym(lat, 3000, v, g, st)
        msg = check_array("out", res["out"], out, "")
        msg = check_array("dv", res["dv"], dv, msg)
        log("  " + check_array("df", res["df"], df, msg))
    else:
        d, n = 8, 1100
        rng = np.random.default_rng(121)
        f = rng.uniform(0, 1, size=(n, d))
        f[:, 0] += 20.0 * np.arange(n)
        f = f.astype(np.float32)
        v = rng.standard_normal((n, 12)).astype(np.float32)
        g = rng.standard_normal((n, 12)).astype(np.float32)
        res = gpu_run(f, v, g, 0)
        olat = O.lattice(f)
        check_filter(res, O, olat, v, g, 0)
