"""Host-side logic of bench.py that needs no GPU: the traffic record lookup, the
algorithmic-byte models and the one-GPU guard."""
import json

import bench


def _write_probe_csv(d, counter, rows):
    """A rocprofv3-style counter CSV: one row per (dispatch, counter)."""
    import csv
    d.mkdir(parents=True)
    with open(d / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            # two rows for one dispatch (per-dimension values are summed)
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": v / 2})
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": v / 2})


def test_probe_summary_from_counter_csv(tmp_path):
    """Sections are cut at the marker dispatches, the copy sets the scales, and every dispatch
    of the step gets its launch name and calibrated bytes."""
    M = "void at::native::bitwise_not_kernel"
    known = bench.calib_known_bytes()
    kib = 1024.0
    fetch = [("warm", 1.0), (M, 0), ("void k_spmm<...>", 100.0), ("void k_gat<...>", 300.0), (M, 0),
             ("copy", known["calib_copy"][0] / 2 / kib), (M, 0), ("read", known["calib_read"][0] / 2 / kib),
             (M, 0), ("g128", known["calib_gather128"][0] / 2 / kib), (M, 0), ("g64", 4096.0), (M, 0),
             ("g32", 4096.0), (M, 0), ("g16", 4096.0), (M, 0)]
    write = [(n, (v / 2 if n not in ("copy",) else known["calib_copy"][1] / kib)) for n, v in fetch]
    _write_probe_csv(tmp_path / "f", "FETCH_SIZE", fetch)
    _write_probe_csv(tmp_path / "w", "WRITE_SIZE", write)
    s = bench.summarize_probe(str(tmp_path / "f"), str(tmp_path / "w"), ["spmm", "gat"])
    assert s["fetch_scale"] == 2.0 and s["write_scale"] == 1.0
    assert [d["launch"] for d in s["step"]] == ["spmm", "gat"]
    g = bench.kernel_traffic(s, "gat")
    assert g["fetch_bytes"] == 300.0 * kib * 2 and g["write_bytes"] == 150.0 * kib
    assert s["step_bytes"] == (100 + 300) * kib * 2 + (50 + 150) * kib
    assert abs(s["calibration"]["calib_read"]["fetch_calibrated_over_known"] - 1.0) < 1e-12
    assert abs(s["calibration"]["calib_gather128"]["fetch_calibrated_over_known"] - 1.0) < 1e-12
    assert bench.kernel_traffic(s, "spmm_t") is None
    # a launch list that does not match the step's dispatches is refused
    import pytest
    with pytest.raises(RuntimeError):
        bench.summarize_probe(str(tmp_path / "f"), str(tmp_path / "w"), ["spmm"])


def test_recorded_traffic_lookup(tmp_path):
    # the committed record either matches the current sources or is ignored
    r = bench.recorded_traffic("skewed_rmat_2400000_hubs")
    assert r is None or r["step_bytes"] > 0
    prof = tmp_path / "profiles"
    prof.mkdir()
    rec = {"source_sha16": bench.library_source_sha(), "fetch_scale": 2.0, "write_scale": 1.0,
           "step": [{"launch": "gat", "kernel": "k", "fetch_bytes": 3.0, "write_bytes": 1.0}], "step_bytes": 4.0}
    (prof / "wl_hbm_traffic.json").write_text(json.dumps(rec))
    r = bench.recorded_traffic("wl", str(prof))
    assert bench.kernel_traffic(r, "gat")["bytes"] == 4.0
    rec["source_sha16"] = "0" * 16                  # stale sources: ignored
    (prof / "wl_hbm_traffic.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("wl", str(prof)) is None


def test_byte_models_match_the_workload_table():
    """The algorithmic-byte models reproduce the figures of the measurement table for the
    workloads' sizes (GB, three significant digits as tabulated)."""
    N5, E5 = 2_400_000, 122_400_000
    assert round(bench.b_spmm(N5, N5, E5, 256, 2, 2) / 1e9, 1) == 64.9
    assert round(bench.b_unique_spmm(N5, N5, E5, 256, 2, 2) / 1e9, 2) == 3.45
    assert round(bench.b_gat(N5, E5, 4, 64, 2, 2, False) / 1e9, 1) == 66.4
    N4, E4 = 2_449_029, 64_308_169
    assert round(bench.b_gat(N4, E4, 8, 16, 4, 4, False) / 1e9, 1) == 36.6
    assert round(bench.b_gat(N4, E4, 8, 16, 4, 4, True) / 1e9, 1) == 38.6
    soft = 4 * (N4 + 1) + 4 * E4 + 4 * N4 * 8 + 8 * E4 * 8
    assert round(soft / 1e9, 2) == 4.46
    assert round(bench.b_spmm(169_343, 169_343, 2_501_829, 128, 4, 4) / 1e9, 3) == 1.388
    assert round(bench.b_spmm(232_965, 232_965, 114_615_892, 256, 4, 4) / 1e9, 1) == 118.5


def test_more_than_one_gpu_is_refused():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_workload_traffic_lookup(tmp_path):
    # the committed per-op record either matches the current library sources or is ignored
    r = bench.recorded_workload_traffic()
    assert r is None or all(v["fetch_bytes"] > 0 and v["write_bytes"] >= 0 for v in r.values())
    prof = tmp_path / "profiles"
    prof.mkdir()
    ops = {"medium_rmat_169343/spmm": {"fetch_bytes": 5.0, "write_bytes": 2.0, "l2_hit": 0.5}}
    rec = {"source_sha16": bench.workloads_source_sha(), "ops": ops}
    (prof / "workloads_1_to_4_hbm_traffic.json").write_text(json.dumps(rec))
    assert bench.recorded_workload_traffic(str(prof)) == ops
    rec["source_sha16"] = "0" * 16
    (prof / "workloads_1_to_4_hbm_traffic.json").write_text(json.dumps(rec))
    assert bench.recorded_workload_traffic(str(prof)) is None


def test_oracle_rate_sampling():
    """The CPU-oracle timer visits each output row at most once, in growing chunks, and
    stops at the budget or when every row is done; whole = one call over everything."""
    seen = []

    def run(sel):
        if sel is None:
            return 100, 10
        seen.extend(sel.tolist())
        return 2 * sel.size, sel.size

    r = bench.oracle_rate(run, 1000, budget_s=60.0, chunk=7)
    assert r["units"] == 1000 and sorted(seen) == list(range(1000))
    assert r["bytes"] == 2000 and r["edges"] == 1000
    seen.clear()
    r = bench.oracle_rate(run, 10**6, budget_s=0.0, chunk=5)   # budget spent after one chunk
    assert r["units"] == 5 and len(set(seen)) == 5
    r = bench.oracle_rate(run, 1000, budget_s=0.0, full=True)
    assert r["units"] == 1000 and r["bytes"] == 100


def test_workloads_probe_summary(tmp_path):
    """Each op's section lies between its own pair of markers; the closing copy scales them."""
    M = "void at::native::bitwise_not_kernel"
    kib = 1024.0
    copy_raw = bench.CALIB_BYTES / 2 / kib
    fetch = [("setup", 9.0), (M, 0), ("k1", 10.0), ("k2", 5.0), (M, 0), ("between", 7.0),
             (M, 0), ("k3", 4.0), (M, 0), (M, 0), ("copy", copy_raw), (M, 0)]
    write = [(n, v / 2) for n, v in fetch]
    _write_probe_csv(tmp_path / "f", "FETCH_SIZE", fetch)
    _write_probe_csv(tmp_path / "w", "WRITE_SIZE", write)
    keys = ["wl/a", "wl/b", "calib_copy"]
    r = bench.summarize_workloads_probe(str(tmp_path / "f"), str(tmp_path / "w"), keys)
    assert set(r) == {"wl/a", "wl/b"}
    assert r["wl/a"]["fetch_bytes"] == 15.0 * kib * 2 and r["wl/b"]["fetch_bytes"] == 4.0 * kib * 2
    assert r["wl/a"]["write_bytes"] == 7.5 * kib * 4      # the copy reads a quarter of its size here
    import pytest
    with pytest.raises(RuntimeError):
        bench.summarize_workloads_probe(str(tmp_path / "f"), str(tmp_path / "w"), keys[:2])


def test_workload_profile_writer(tmp_path):
    """--summarize-workloads: the per-op record the workload lines fall back on, stamped with the
    sources' hash, read back by recorded_workload_traffic."""
    M = "void at::native::bitwise_not_kernel"
    kib = 1024.0
    copy_raw = bench.CALIB_BYTES / 2 / kib
    fetch = [(M, 0), ("k1", 10.0), (M, 0), (M, 0), ("copy", copy_raw), (M, 0)]
    _write_probe_csv(tmp_path / "f", "FETCH_SIZE", fetch)
    _write_probe_csv(tmp_path / "w", "WRITE_SIZE", [(n, v) for n, v in fetch])
    probe = tmp_path / "probe.json"
    probe.write_text(json.dumps({"keys": ["wl/spmm", "calib_copy"]}))
    out = tmp_path / "profiles"
    out.mkdir()
    bench.write_workload_profile(str(tmp_path / "f"), str(tmp_path / "w"), str(probe), str(out))
    ops = bench.recorded_workload_traffic(str(out))
    assert ops["wl/spmm"]["fetch_bytes"] == 10.0 * kib * 2
    assert (out / "workloads_1_to_4_hbm_counters.txt").read_text().count("wl/spmm") == 1


def test_stats_profile_writer(tmp_path):
    """--summarize-stats: kernels ordered by total time, durations in ms, the command recorded."""
    import argparse
    d = tmp_path / "stats"
    d.mkdir()
    (d / "run_kernel_stats.csv").write_text(
        '"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
        '"void cogdl::k_a<int>(cogdl::X)",2,3000000,1500000.0,25.0,1000000,2000000,1.0\n'
        '"void cogdl::k_b<int>(cogdl::X)",3,9000000,3000000.0,75.0,2000000,4000000,1.0\n')
    out = tmp_path / "profiles"
    out.mkdir()
    bench.write_stats_profile(argparse.Namespace(config=5), str(d), "the command", str(out))
    txt = (out / "skewed_rmat_2400000_hubs_kernel_stats.txt").read_text().splitlines()
    assert txt[1] == "# command: the command"
    body = [l for l in txt if not l.startswith("#")][1:]
    assert body[0].startswith("void k_b<int>") and "3.0000" in body[0]
    assert body[1].startswith("void k_a<int>")


def test_plans_profile_writer(tmp_path):
    """--summarize-plans: the two runs' lines side by side, refused for different workloads."""
    import pytest

    def line(step, wl="wl_a: graph"):
        return {"ms_per_step": step, "value": 1000.0 / step, "config": {"workload": wl},
                "ops": {"spmm": {"ms": step / 4}}, "kernels": {"spmm": {"avg_ms": step / 5}, "fill": {"avg_ms": 1.0}},
                "ops_outside_step": {"sddmm_edge_softmax": {"ms": 2.0}},
                "inference": {"gcn": {"ms": 3.0}}, "roofline": {"kernel": "spmm", "avg_ms": step / 5}}
    a, b = tmp_path / "a.json", tmp_path / "b.json"
    a.write_text("[bench] log line\n" + json.dumps(line(20.0)))
    b.write_text(json.dumps(line(25.0)))
    out = tmp_path / "profiles"
    out.mkdir()
    bench.write_plans_profile(str(a), str(b), str(out))
    txt = (out / "wl_a_sliced_vs_plain.txt").read_text()
    assert "step ms (timed region)" in txt and "20.000" in txt and "25.000" in txt
    assert "kernel spmm ms" in txt and "kernel fill" not in txt and "inference GCN ms" in txt
    b.write_text(json.dumps(line(25.0, "wl_b: other")))
    with pytest.raises(SystemExit):
        bench.write_plans_profile(str(a), str(b), str(out))
