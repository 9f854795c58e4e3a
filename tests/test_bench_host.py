"""Host logic of bench.py (no GPU): the minimum-traffic byte model and the
counter summaries (rocprofv3 CSVs -> per-kernel figures)."""
import csv
import json

import bench


def test_step_bytes_model():
    """N(16d + 20C) + M(8 + 8(d+1)) + 16MC bytes per build + forward +
    backward step; the forward-only variant N(8d + 8C) + ... + 8MC."""
    n, d, C, M = 2_097_152, 5, 32, 21_133
    assert bench.step_bytes(n, d, C, M) == n * (16 * d + 20 * C) + M * (8 + 8 * (d + 1)) + 16 * M * C
    assert bench.step_bytes(n, d, C, M, forward_only=True) == n * (8 * d + 8 * C) + M * (8 + 8 * (d + 1)) + 8 * M * C
    # per-launch model: the splat reads f and v and writes the lattice once
    assert bench.kernel_bytes("splat", n, d, C, M) == 4 * d * n + 4 * C * n + 4 * M * C


def _write_csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value", "Grid_Size"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_counter_summary_takes_main_instance_and_calibration(tmp_path, monkeypatch):
    """Per kernel, the dispatches of its most-dispatched template instance
    (not the small d=3 check in the same run), scaled by the known bytes of
    the calibration copy (FETCH x2 here, WRITE x1)."""
    monkeypatch.setattr(bench, "source_hash", lambda: "test")
    big, small = "void pam::k_splat<5, 4, 0, 32, false>(args)", "void pam::k_splat<3, 4, 0, 8, false>(args)"
    copy = "__amd_rocclr_copyBuffer"
    mib = 512
    fetch = [{"Kernel_Name": copy, "Counter_Name": "FETCH_SIZE", "Counter_Value": mib * 1024 / 2, "Grid_Size": 99}]
    write = [{"Kernel_Name": copy, "Counter_Name": "WRITE_SIZE", "Counter_Value": mib * 1024, "Grid_Size": 99}]
    for v in (100.0, 110.0, 120.0):
        fetch.append({"Kernel_Name": big, "Counter_Name": "FETCH_SIZE", "Counter_Value": v, "Grid_Size": 4096})
        write.append({"Kernel_Name": big, "Counter_Name": "WRITE_SIZE", "Counter_Value": v / 10, "Grid_Size": 4096})
    fetch.append({"Kernel_Name": small, "Counter_Name": "FETCH_SIZE", "Counter_Value": 1.0, "Grid_Size": 4})
    write.append({"Kernel_Name": small, "Counter_Name": "WRITE_SIZE", "Counter_Value": 1.0, "Grid_Size": 4})
    fp, wp, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "t.json"
    _write_csv(fp, fetch)
    _write_csv(wp, write)
    rec = bench.summarize_counters(str(fp), str(wp), mib, str(out))
    k = rec["kernels"]["k_splat"]
    assert k["dispatches"] == [3, 3]
    assert abs(rec["fetch_scale"] - 2.0) < 1e-12 and abs(rec["write_scale"] - 1.0) < 1e-12
    assert abs(k["fetch_bytes"] - 110.0 * 2 * 1024) < 1e-6
    assert abs(k["write_bytes"] - 11.0 * 1024) < 1e-6
    assert json.load(open(out))["source_sha256_16"] == "test"


def test_pmc_summary_takes_main_instance(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "source_hash", lambda: "test")
    big, small = "void pam::k_slice<5, 4, 32>(args)", "void pam::k_slice<3, 4, 8>(args)"
    rows = [{"Kernel_Name": big, "Counter_Name": "SQ_WAVES", "Counter_Value": v, "Grid_Size": 1} for v in (8, 10)]
    rows.append({"Kernel_Name": small, "Counter_Name": "SQ_WAVES", "Counter_Value": 1000, "Grid_Size": 1})
    p = tmp_path / "p.csv"
    _write_csv(p, rows)
    rec = bench.summarize_pmc([str(p)], str(tmp_path / "c.json"))
    assert rec["kernels"]["k_slice"]["SQ_WAVES"] == 9.0
