#!/usr/bin/env python3
"""Throughput of the permutohedral-lattice filter (build + forward + backward)
on one MI355X, as one JSON line.

A step is one pass of the whole path over one synthetic volume: lattice
build (embedding, hash insert, compaction, per-point vertex ids, neighbour
table), forward filter (splat, d+1 blur passes, slice) and backward filter
(splat of the upstream gradient, d+1 reversed blur passes, slice of the value
gradient plus the embedding gradient).  Inputs are resident in HBM before the
timed region starts.

Default workload: 128x128x128 voxels (N = 2,097,152), d = 5 (coordinates/16
plus two mixture channels), C = 32 value channels, raw (unnormalised) mode.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published
METRIC = "Mvoxels/s PAM lattice filter fwd+bwd, 128³ d=5 C=32; % HBM roofline"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_C3.json")
PMC_FILE = os.path.join(ROOT, "profiles", "counters_C3.json")
KERNEL_SRCS = [os.path.join(ROOT, "paper_1907_00641_amd", "csrc", f)
               for f in ("pam_device.h", "pam_build.hip", "pam_filter.hip")]


def kernel_bytes(name: str, n: int, d: int, C: int, M: int, ldq: int = 0) -> float:
    """Algorithmic bytes of one launch under the minimum-traffic model: the
    arrays the kernel's contract must read once and write once, with the
    simplex source counted as the n x d features (4d bytes per point) and
    the lattice at its C channels (4MC bytes).  Cached per-point records,
    vertex ids, the permutation and tile lists are extra traffic, not part
    of the model; the build's kernels are accounted as one stage
    (``build_bytes``)."""
    src = 4 * d * n          # simplex source (features), once per call
    row = 4 * C * n          # one n x C array
    lat = 4 * M * C          # one lattice buffer
    latq = 4 * M * ldq       # one augmented-channel lattice buffer (d*C channels)
    table = {
        "splat": src + row + lat,                 # reads f and v, writes L once
        "splat_bwd": src + row + lat,             # reads f and g, writes L once
        "slice": src + lat + row,                 # reads f and A once, writes out
        "slice_bwd": 2 * src + 3 * row + 2 * lat,  # reads f, v, g, A, At; writes dv, df
        "splat_aug": src + row + latq,
        "slice_aug": 2 * src + 2 * row + 2 * lat + 2 * latq,
    }
    return float(table.get(name, 0.0))


def blur_bytes(M: int, C: int, d: int, directions: float) -> float:
    """One blur launch over `directions` lattice directions: the lattice read
    once and written once, plus the directions' neighbour ids."""
    return float(2 * 4 * M * C + 8 * M * directions)


def build_bytes(n: int, d: int, M: int) -> float:
    """The build stage: reads f once, writes the vertex keys (8 B) and the
    neighbour table (2 ids per direction)."""
    return float(4 * d * n + 8 * M + 8 * M * (d + 1))


def step_bytes(n: int, d: int, C: int, M: int, augmented: bool = False, forward_only: bool = False) -> float:
    """Minimum traffic of one build + fwd + bwd step: the build reads f, the
    forward reads the simplex source and v and writes out, the backward
    reads the simplex source, g and v and writes dv and df: 16d + 20C bytes
    per point (build + forward only: 8d + 8C); plus the lattice: keys and
    neighbours written once, each filter's lattice written once and read
    once.  The augmented-channel gradient adds two lattices of d*C channels
    written and read once."""
    if forward_only:
        return float(n * (8 * d + 8 * C) + M * (8 + 8 * (d + 1)) + 8 * M * C)
    b = n * (16 * d + 20 * C) + M * (8 + 8 * (d + 1)) + 2 * 8 * M * C
    if augmented:
        b += 2 * 8 * M * d * C
    return float(b)


def source_hash() -> str:
    """Hash of the kernel sources; counter readings are only valid for it."""
    h = hashlib.sha256()
    for path in KERNEL_SRCS:
        with open(path, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_counters(path: str):
    """A committed per-kernel counter summary (profiles/*.json written by
    --summarize-counters / --summarize-pmc), or None when it is absent or was
    taken on other kernel sources."""
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256_16") != source_hash():
        return None
    return rec.get("kernels", {})


def host_info() -> dict:
    """Logical CPUs of the host and its CPU model (from /proc/cpuinfo)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model}


def cpu_baseline(data, d: int, C: int, flags: int, min_seconds: float = 10.0, group_start=None,
                 augmented: bool = False, asym_keys=None):
    """The oracle, untuned and single-threaded C, on the same volume(s):
    build + forward + backward (each group on its own) repeated until at
    least ``min_seconds`` of CPU work have run."""
    from oracle import oracle as O

    norm = bool(flags & 1)
    n = data["f"].shape[0]
    gs = group_start if group_start is not None else [0, n]
    reps, total = 0, 0.0
    while total < min_seconds:
        t0 = time.perf_counter()
        if asym_keys is not None:
            lat = O.lattice(data["f"])
            out, st = O.forward_asym(lat, asym_keys, data["v"])
            O.backward_asym(lat, asym_keys, data["v"], data["g"], st)
            total += time.perf_counter() - t0
            reps += 1
            continue
        for a, e in zip(gs[:-1], gs[1:]):
            lat = O.lattice(data["f"][a:e])
            out, st = O.forward(lat, data["v"][a:e], norm)
            O.backward(lat, data["v"][a:e], data["g"][a:e], norm, st)
            if augmented:
                O.backward_augmented(lat, data["f"][a:e], data["v"][a:e], data["g"][a:e])
        total += time.perf_counter() - t0
        reps += 1
    what = f"the whole {n}-voxel volume" if len(gs) == 2 else f"all {len(gs) - 1} volumes ({n} voxels)"
    return {"value": n * reps / total / 1e6, "unit": "Mvoxels/s", "cores": 1, "kind": "oracle",
            "sample": f"{what}, build + fwd + bwd {reps} times in {total:.1f} s, single thread",
            "threads_used": 1, **host_info()}


def main_instances(inst: dict) -> dict:
    """Per kernel symbol (template arguments dropped), the dispatches of its
    most-dispatched template instance: the benchmark's own workload, not the
    small d=3 approximation check that runs in the same process."""
    best = {}
    for name, vals in inst.items():
        short = name.replace("void ", "").replace("pam::", "").split("<")[0]
        if short not in best or len(vals) > len(best[short]):
            best[short] = vals
    return best


def summarize_counters(fetch_csv: str, write_csv: str, calib_mb: int, out_path: str) -> dict:
    """Turn two rocprofv3 --pmc runs of this script (FETCH_SIZE, then
    WRITE_SIZE; KiB per dispatch) into HBM bytes per launch of each kernel.
    Each counter is scaled by the ratio of the known bytes of the plain
    device copy that ``--copy-calibration-mb`` runs first (the largest copy
    dispatch) to what the same counter reads for it."""
    import csv
    from collections import defaultdict

    def load(path, counter):
        inst, copy = defaultdict(list), []
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                name = r["Kernel_Name"]
                val = float(r["Counter_Value"])
                if "copyBuffer" in name:
                    copy.append((int(r["Grid_Size"]), val))
                elif name.startswith(("void pam::", "pam::")):
                    inst[name.split("(")[0]].append(val)
        return main_instances(inst), max(copy)[1] if copy else None

    known_kib = float(calib_mb) * 1024.0
    fetch, fcopy = load(fetch_csv, "FETCH_SIZE")
    write, wcopy = load(write_csv, "WRITE_SIZE")
    if not fcopy or not wcopy:
        raise SystemExit("no calibration copy dispatch in the counter runs")
    fs, ws = known_kib / fcopy, known_kib / wcopy
    kernels = {}
    for k in sorted(set(fetch) & set(write)):
        f_kib = sum(fetch[k]) / len(fetch[k])
        w_kib = sum(write[k]) / len(write[k])
        kernels[k] = {"fetch_bytes": f_kib * fs * 1024, "write_bytes": w_kib * ws * 1024,
                      "bytes_per_launch": (f_kib * fs + w_kib * ws) * 1024,
                      "dispatches": [len(fetch[k]), len(write[k])]}
    rec = {"source_sha256_16": source_hash(), "fetch_scale": fs, "write_scale": ws,
           "calibration": f"device copy of {calib_mb} MiB: FETCH_SIZE {fcopy:.0f} KiB, WRITE_SIZE {wcopy:.0f} KiB",
           "kernels": kernels}
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
    return rec


def summarize_pmc(csvs, out_path: str) -> dict:
    """Per-kernel averages over dispatches of every counter in rocprofv3
    --pmc CSVs of this script (the filter's kernels only, each kernel's
    most-dispatched template instance), with the hash of the kernel sources
    they were taken on."""
    import csv
    from collections import defaultdict

    acc = defaultdict(lambda: defaultdict(list))  # counter -> template instance -> values
    for path in csvs:
        with open(path) as fh:
            for r in csv.DictReader(fh):
                name = r["Kernel_Name"]
                if not name.startswith(("void pam::", "pam::")):
                    continue
                acc[r["Counter_Name"]][name.split("(")[0]].append(float(r["Counter_Value"]))
    kernels = defaultdict(dict)
    for counter, inst in acc.items():
        for k, v in main_instances(inst).items():
            kernels[k][counter] = sum(v) / len(v)
    kernels = dict(kernels)
    rec = {"source_sha256_16": source_hash(), "kernels": kernels}
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    return rec


def approximation_error(P, torch) -> dict:
    """The lattice filter against the exact Gaussian sum it approximates
    (eq. 4-5 with the kernel exp(-|f_i - f_j|^2 / 2)) on the 12^3 corner of
    the 32^3 d=3 workload (N = 1728): relative L2 error of the GPU output in
    raw and normalised mode, and the least-squares gain of the raw output
    against the exact sum.  The exact sum is evaluated here in fp64 numpy."""
    import numpy as np

    import synth

    data = synth.generate("C1", shape=(12, 12, 12))
    f, v = data["f"].astype(np.float64), data["v"].astype(np.float64)
    sq = np.sum(f * f, axis=1)
    k = np.exp(-0.5 * np.maximum(sq[:, None] + sq[None, :] - 2.0 * f @ f.T, 0.0))
    exact = k @ v
    exact_norm = exact / k.sum(axis=1, keepdims=True)
    dev = torch.device("cuda:0")
    ft, vt = torch.from_numpy(data["f"]).to(dev), torch.from_numpy(data["v"]).to(dev)
    lat = P.pam_lattice_build(ft)
    raw = P.pam_filter_fwd(lat, vt, 0).cpu().numpy().astype(np.float64)
    nrm = P.pam_filter_fwd(lat, vt, 1).cpu().numpy().astype(np.float64)
    lat.destroy()

    def rel(a, b):
        return float(np.linalg.norm(a - b) / np.linalg.norm(b))

    gain = float(np.sum(raw * exact) / np.sum(raw * raw))
    return {"points": int(f.shape[0]), "d": int(f.shape[1]), "C": int(v.shape[1]),
            "rel_l2_raw": rel(raw, exact), "rel_l2_normalized": rel(nrm, exact_norm),
            "G_fit_over_G_d": 1.0 / gain}


def row_ceiling(x, torch, P, reps: int = 10) -> dict:
    """HBM ceilings of the per-point kernels' access pattern, measured with
    the library's row-copy probe on the n x C value array: rows copied in
    order, read from a random permutation, written to one, or both (GB/s of
    bytes moved).  The per-point filter kernels read and write value rows at
    the original index of points taken in the simplex-sorted order, i.e. at
    random rows."""
    n, c = x.shape
    gen = torch.Generator(device=x.device)
    gen.manual_seed(1907)
    perm = torch.randperm(n, device=x.device, generator=gen).to(torch.int32)
    y = torch.empty_like(x)
    rows = 2.0 * x.numel() * x.element_size()
    res = {}
    for mode, name in enumerate(("sequential", "random_read", "random_write", "random_both")):
        nbytes = rows + (perm.numel() * 4 if mode else 0)
        P.pam_probe_copy_rows(x, y, perm, mode)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            P.pam_probe_copy_rows(x, y, perm, mode)
        b.record()
        torch.cuda.synchronize()
        res[f"{name}_GBs"] = nbytes / (a.elapsed_time(b) / reps * 1e-3) / 1e9
    res["row_bytes"] = c * x.element_size()
    res["rows"] = n
    del y, perm
    return res


KERNEL_SYMBOL = {  # timing kind -> kernel symbol (without template arguments)
    "range": "k_range", "layout": "k_layout", "fill": "k_fill_f32", "insert": "k_insert_tiles",
    "compact": "k_compact", "resolve": "k_resolve", "scan": "k_scan_lds", "scatter": "k_scatter",
    "tiles": "k_sorted_tiles", "splat": "k_splat", "splat_bwd": "k_splat", "blur": "k_blur2", "slice": "k_slice",
    "slice_bwd": "k_slice_bwd", "splat_aug": "k_splat", "slice_aug": "k_slice_aug",
}


BLOCK = {"dims": (80, 80, 48), "c_in": 18, "d_tot": 10, "c_tot": 16, "groups": 2, "mesh_scale": 1.0 / 8.0,
         "slope": 0.01}


def block_inputs(cfg, seed: int = 1907900):
    """Input channels i.i.d. N(0, 1); weights N(0, 1/fan_in), biases N(0, 0.1^2); upstream gradient of
    the block's grouped output N(0, 1)."""
    import numpy as np

    rng = np.random.default_rng(seed)
    W, H, D = cfg["dims"]
    n = W * H * D
    c_in, d_tot, c_tot = cfg["c_in"], cfg["d_tot"], cfg["c_tot"]
    x = rng.standard_normal((n, c_in)).astype(np.float32)
    wf = (rng.standard_normal((d_tot, c_in + 3)) / np.sqrt(c_in + 3)).astype(np.float32)
    bf = (0.1 * rng.standard_normal(d_tot)).astype(np.float32)
    wv = (rng.standard_normal((c_tot, c_in)) / np.sqrt(c_in)).astype(np.float32)
    bv = (0.1 * rng.standard_normal(c_tot)).astype(np.float32)
    gout = rng.standard_normal((n * cfg["groups"], c_tot // cfg["groups"])).astype(np.float32)
    return x, wf, bf, wv, bv, gout


def cpu_baseline_block(cfg, arrs, min_seconds: float = 10.0):
    """The oracle chain of the block (prologue, each group's lattice,
    filter, backward, prologue backward), single thread, repeated until at
    least min_seconds."""
    import numpy as np

    from oracle import block as OB
    from oracle import oracle as O

    x, wf, bf, wv, bv, gout = arrs
    dims, G = cfg["dims"], cfg["groups"]
    n = dims[0] * dims[1] * dims[2]
    reps, total = 0, 0.0
    while total < min_seconds:
        t0 = time.perf_counter()
        f, v = OB.prologue_fwd(x, dims, wf, bf, wv, bv, cfg["mesh_scale"], cfg["slope"], G)
        f32 = f.astype(np.float32)
        df, dv = np.zeros_like(f), np.zeros_like(v)
        for g in range(G):
            s = slice(g * n, (g + 1) * n)
            lat = O.lattice(f32[s])
            _, st = O.forward(lat, v[s], False)
            dv[s], df[s] = O.backward(lat, v[s], gout[s], False, st)
        OB.prologue_bwd(x, dims, wf, bf, wv, cfg["mesh_scale"], cfg["slope"], G, df, dv)
        total += time.perf_counter() - t0
        reps += 1
    return {"value": n * reps / total / 1e6, "unit": "Mvoxels/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole {n}-voxel block, {reps} times in {total:.1f} s, single thread",
            "threads_used": 1, **host_info()}


def bench_block(args) -> int:
    import torch

    import paper_1907_00641_amd as P

    cfg = BLOCK
    arrs = block_inputs(cfg)
    dev = torch.device("cuda:0")
    x, wf, bf, wv, bv, gout = (torch.from_numpy(a).to(dev) for a in arrs)
    W, H, D = cfg["dims"]
    n, G = W * H * D, cfg["groups"]
    desc = P.block_desc(cfg["c_in"], cfg["d_tot"], cfg["c_tot"], G, cfg["dims"], cfg["mesh_scale"], cfg["slope"])
    gs = [g * n for g in range(G + 1)]
    lat = None

    def step():
        nonlocal lat
        feat, val = P.pam_block_fwd(desc, x, wf, bf, wv, bv)
        lat = P.pam_lattice_build(feat, lat=lat, group_start=gs)
        P.pam_filter_fwd(lat, val)
        dval, dfeat = P.pam_filter_bwd(lat, val, gout)
        P.pam_block_bwd(desc, x, wf, bf, wv, dfeat, dval)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    M, _ = P.pam_lattice_stats(lat)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    rec = {"metric": "Mvoxels/s permutohedral block (prologue, PAM fwd+bwd over 2 groups, prologue bwd), 80x80x48",
           "value": n / (ms * 1e-3) / 1e6, "unit": "Mvoxels/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": "U-PAM-Net half-resolution block: 80x80x48 voxels, 18 input channels, "
                                  "2 groups of d=5 features and C=8 descriptors", "voxels": n, "M": M, **{
                                      k: v for k, v in cfg.items() if k != "dims"}}}
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline_block(cfg, arrs)
    lat.destroy()
    print(json.dumps(rec), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="C3")
    ap.add_argument("--normalize", action="store_true")
    ap.add_argument("--block", action="store_true",
                    help="the whole permutohedral block at U-PAM-Net's half resolution (80x80x48): 1x1x1 "
                         "feature/descriptor prologue (18 input channels, mesh, Leaky-ReLU), two channel groups "
                         "(d = 5, C = 8 each) in one batched build, filter forward and backward, prologue backward")
    ap.add_argument("--asym", action="store_true",
                    help="asymmetric filter: the volume's voxels are the keys, the same voxels moved by half a "
                         "voxel along each spatial axis the queries (one lattice over both; raw mode)")
    ap.add_argument("--egrad", choices=("eq8", "augmented"), default="eq8",
                    help="embedding gradient: eq. 8 (default) or the augmented-channel estimator (raw mode)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run one plain device copy of this many MiB first (untimed), so that "
                         "rocprofv3 counter runs can scale FETCH_SIZE/WRITE_SIZE against known bytes")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the traffic summary from two rocprofv3 counter CSVs and exit")
    ap.add_argument("--traffic-out", default=TRAFFIC_FILE)
    ap.add_argument("--summarize-pmc", nargs="+", metavar="PMC_CSV",
                    help="write the per-kernel counter summary from rocprofv3 --pmc CSVs and exit")
    ap.add_argument("--pmc-out", default=PMC_FILE)
    args = ap.parse_args(argv)
    if args.summarize_counters:
        rec = summarize_counters(*args.summarize_counters, args.copy_calibration_mb or 512, args.traffic_out)
        print(json.dumps({k: round(v["bytes_per_launch"]) for k, v in rec["kernels"].items()}))
        return 0
    if args.summarize_pmc:
        rec = summarize_pmc(args.summarize_pmc, args.pmc_out)
        print(json.dumps(rec["kernels"]))
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the lattice filter runs on one device; see the sharding design notes)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_1907_00641_amd as P
    import synth

    if not torch.cuda.is_available():
        print("no GPU available", file=sys.stderr)
        return 1
    if args.block:
        return bench_block(args)
    w = synth.WORKLOADS[args.workload]
    flags = 1 if args.normalize else 0
    augmented = args.egrad == "augmented"
    if augmented and flags:
        print("the augmented-channel embedding gradient is raw mode only", file=sys.stderr)
        return 2
    bwd_flags = flags | (P.PAM_EGRAD_AUGMENTED if augmented else 0)
    if args.asym and (flags or augmented or w.batch != 1):
        print("the asymmetric filter is timed in raw mode with the eq. 8 gradient on one volume", file=sys.stderr)
        return 2
    group_start = None
    if w.batch == 1:
        data = synth.generate(w)
    else:  # a batch of volumes: one batched build, each volume its own point group
        vols = [synth.generate(w, volume=b) for b in range(w.batch)]
        data = {k: np.concatenate([x[k] for x in vols]) for k in ("f", "v", "g")}
        group_start = np.cumsum([0] + [x["f"].shape[0] for x in vols]).tolist()
    n_keys = data["f"].shape[0]
    if args.asym:  # keys, then the same voxels moved by half a voxel (coordinates are the first 3 channels)
        fq = data["f"].copy()
        fq[:, :3] += np.float32(0.5 / w.sigma_s)
        data = {"f": np.concatenate([data["f"], fq]), "v": data["v"], "g": data["g"]}
    n, d = data["f"].shape
    C = data["v"].shape[1]
    dev = torch.device("cuda:0")
    f, v, g = (torch.from_numpy(data[k]).to(dev) for k in ("f", "v", "g"))
    out = torch.empty_like(g)
    dv = torch.empty_like(v)
    df = torch.empty_like(f)
    stream = torch.cuda.current_stream()
    if args.copy_calibration_mb > 0:
        nbytes = args.copy_calibration_mb << 20
        src = torch.ones(nbytes // 4, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)  # reads and writes exactly nbytes each
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()

    lat = None

    def step(ev=None):
        nonlocal lat
        lat = P.pam_lattice_build(f, lat=lat, group_start=group_start)
        if ev:
            ev[1].record(stream)
        if args.asym:
            P.pam_filter_fwd_asym(lat, n_keys, v, out=out)
            if ev:
                ev[2].record(stream)
            P.pam_filter_bwd_asym(lat, n_keys, v, g, grad_val=dv, grad_feat=df)
            return
        P.pam_filter_fwd(lat, v, flags, out=out)
        if ev:
            ev[2].record(stream)
        P.pam_filter_bwd(lat, v, g, bwd_flags, grad_val=dv, grad_feat=df)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    M, cap = P.pam_lattice_stats(lat)

    # headline: K whole steps, no instrumentation
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps

    # per-stage durations: events around the build, the forward and the
    # backward call of each of K more steps; medians
    evs = []
    for _ in range(args.steps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        step(e)
        e[3].record(stream)
        evs.append(e)
    torch.cuda.synchronize()
    stage = {"build": [], "fwd": [], "bwd": [], "sum": []}
    for e in evs:
        tb, tf, tw = e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])
        stage["build"].append(tb)
        stage["fwd"].append(tf)
        stage["bwd"].append(tw)
        stage["sum"].append(tb + tf + tw)
    stages = {f"t_{k}_ms_median": float(np.median(v)) for k, v in stage.items()}

    # per-kernel durations: HIP events recorded by the library around each
    # of its launches, on the stream the kernels run on, over K more steps
    P.pam_timing_enable(lat, True)
    for _ in range(args.steps):
        step()
    per_kernel = P.pam_timing_read(lat)
    P.pam_timing_enable(lat, False)
    torch.cuda.synchronize()

    ceiling = row_ceiling(v, torch, P)

    ldq = (d * C + 3) // 4 * 4     # augmented-channel lattice row stride
    # the committed counter runs are of the default workload (C3, raw mode,
    # eq. 8 gradient, symmetric): other workloads report no counters
    default_run = w.name == "C3" and not flags and not augmented and not args.asym
    traffic = load_counters(TRAFFIC_FILE) if default_run else None
    pmc = load_counters(PMC_FILE) if default_run else None
    kernels = {}
    for name, (cnt, ms) in per_kernel.items():
        avg_ms = ms / cnt
        per_step = cnt / args.steps
        if name == "blur":
            b = blur_bytes(M, C, d, (d + 1) / per_step)
        else:
            b = kernel_bytes(name, n, d, C, M, ldq)
        sym = KERNEL_SYMBOL.get(name, name)
        kr = {"symbol": sym, "launches_per_step": per_step, "avg_us": avg_ms * 1e3, "ms_per_step": ms / args.steps,
              "algorithmic_bytes_per_launch": b or None,
              "algorithmic_GBs": (b / (avg_ms * 1e-3) / 1e9) if b else None}
        if traffic and sym in traffic:
            kr["counter_bytes_per_launch"] = traffic[sym]["bytes_per_launch"]
        kernels[name] = kr
    # the dominant kernel: the symbol with the largest share of the step
    # (both splat launches are one kernel)
    by_sym = {}
    for name, kr in kernels.items():
        by_sym.setdefault(kr["symbol"], []).append(name)
    dom_sym = max(by_sym, key=lambda k: sum(kernels[x]["ms_per_step"] for x in by_sym[k]))
    dom = by_sym[dom_sym]
    dom_launches = sum(kernels[x]["launches_per_step"] for x in dom)
    dom_ms = sum(kernels[x]["ms_per_step"] for x in dom)
    dom_avg_us = dom_ms / dom_launches * 1e3
    dom_bytes = sum((kernels[x]["algorithmic_bytes_per_launch"] or 0.0) * kernels[x]["launches_per_step"]
                    for x in dom) / dom_launches
    achieved = dom_bytes / (dom_avg_us * 1e-6) / 1e9
    dom_traffic = traffic[dom_sym]["bytes_per_launch"] if traffic and dom_sym in traffic else None
    sbytes = step_bytes(n, d, C, M, augmented)
    step_gbs = sbytes / (ms_per_step * 1e-3) / 1e9
    # whole-step counter traffic (HBM bytes from FETCH_SIZE + WRITE_SIZE of
    # every launch of the step) over the uninstrumented step time
    step_counter = None
    if traffic:
        tot = 0.0
        for name, kr in kernels.items():
            sym = kr["symbol"]
            if sym in traffic:
                tot += traffic[sym]["bytes_per_launch"] * kr["launches_per_step"]
        step_counter = {"bytes_per_step": tot, "GBs": tot / (ms_per_step * 1e-3) / 1e9,
                        "frac": tot / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, "over_bytes_min": tot / sbytes}
    counters = None
    if pmc:
        counters = {}
        for sym, cs in pmc.items():
            counters[sym] = {k: cs[k] for k in ("TCC_ATOMIC_sum", "TCP_TCC_ATOMIC_WITHOUT_RET_REQ_sum",
                                                 "SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS") if k in cs}

    rec = {
        "metric": (METRIC if w.name == "C3" and not augmented and not args.asym else
                   f"Mpoints/s asymmetric PAM lattice filter fwd+bwd (keys + queries), {w.name}" if args.asym else
                   f"Mvoxels/s PAM lattice filter fwd+bwd, {w.name}" + (", augmented-channel embedding gradient"
                                                                       if augmented else "")),
        "value": n / (ms_per_step * 1e-3) / 1e6,
        "unit": "Mvoxels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}", "voxels": n, "d": d, "C": C, "M": M, "groups": w.batch,
                   "mode": "normalized" if flags else "raw", "embedding_gradient": args.egrad,
                   "asymmetric": bool(args.asym), "keys": n_keys if args.asym else None,
                   "table_capacity": cap},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": dom_traffic, "kernel": dom_sym,
                     "kernel_calls": dom, "launches_per_step": dom_launches, "kernel_avg_us": dom_avg_us,
                     "algorithmic_bytes_per_launch": dom_bytes},
        "step_roofline": {"bytes_min": sbytes, "achieved_GBs": step_gbs, "frac": step_gbs / PEAK_HBM_GBS,
                          "counter_traffic": step_counter},
        "stages": stages,
        "kernels": kernels,
        "counters": counters,
        "ceiling": ceiling,
    }
    if not args.asym and w.name == "C3":
        rec["approximation"] = approximation_error(P, torch)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(data, d, C, flags, group_start=group_start, augmented=augmented,
                                           asym_keys=n_keys if args.asym else None)
    lat.destroy()
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
