"""Host-side logic of bench.py that needs no GPU: the traffic record lookup, the
algorithmic-byte models and the one-GPU guard."""
import json

import bench


def test_recorded_traffic_lookup(tmp_path):
    # the committed record either matches the current sources or is ignored
    for k in bench.ROOFLINE_KERNELS:
        r = bench.recorded_traffic("skewed_rmat_2400000_hubs", k)
        assert r is None or r["bytes"] > 0
    # a record written for the current sources is found at the timed step's dispatch
    prof = tmp_path / "profiles"
    prof.mkdir()
    spec = bench.ROOFLINE_KERNELS["spmm_t"]
    disp = [{"fetch_bytes": 10.0 * i, "write_bytes": 1.0, "dur_ms": 0.1} for i in range(6)]
    rec = {"source_sha16": {k: bench.kernel_source_sha(k) for k in bench.ROOFLINE_KERNELS},
           "warmup": 1, "kernels": {spec["name"]: disp}}
    (prof / "wl_hbm_traffic.json").write_text(json.dumps(rec))
    r = bench.recorded_traffic("wl", "spmm_t", str(prof))
    assert r["dispatch"] == 3 and r["bytes"] == 31.0
    # stale sources: ignored
    rec["source_sha16"]["spmm_t"] = "0" * 16
    (prof / "wl_hbm_traffic.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("wl", "spmm_t", str(prof)) is None


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
