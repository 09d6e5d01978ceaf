"""Host-side logic of bench.py that needs no GPU: the traffic record lookup."""
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
