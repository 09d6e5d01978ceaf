#!/usr/bin/env python3
"""Benchmark of the GNN message-passing hot path on one MI355X.

One step is one pass of the whole path over the skewed R-MAT workload
(2,400,000 nodes, 120,000,000 distinct edges plus self-loops = 122,400,000
nonzeros, four planted hub rows of 100k-300k edges, bf16 features with fp32
accumulation):

  a1  balancer (plan rebuild) on the CSR
  a2  SpMM   Y  = A X           X bf16 [N, 256] -> Y bf16
  a3  CSR -> CSC transpose (stable, with perm)
  a1  balancer on the CSC
  a4  SpMM^T dX = A^T G         G bf16 [N, 256] -> dX bf16
  a5-a7 fused GAT aggregation: scores -> LeakyReLU -> edge softmax -> 4 x 64 bf16 SpMM

Inputs are resident in HBM before the timed region.  The value is the
effective HBM bandwidth of the step: algorithmic bytes (what the method must
move, one gather of a feature row per nonzero) divided by the step time.
Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0
SLICE_MIN = 128          # COGDL_DEFAULT_SLICE_MIN: rows longer than this are column-sliced
METRIC = "SpMM & GAT-aggregate effective HBM GB/s (% of peak) and edges/sec, 1 MI355X"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload number (default: the skewed R-MAT)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="CPU-baseline time budget")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-inference", action="store_true",
                    help="skip the 2-layer GCN / GAT inference timing on the Reddit-shaped graph")
    ap.add_argument("--group-size", type=int, default=0)
    ap.add_argument("--plain-plans", action="store_true",
                    help="balancer plans without column slicing (the paper's neighbour groups only)")
    ap.add_argument("--alpha-out", action="store_true",
                    help="also write alpha in the GAT step (takes the given-scores entry point)")
    ap.add_argument("--gat-scores", choices=("proj", "given"), default="proj",
                    help="GAT step: source scores projected from the gathered feature rows "
                         "(cogdl_gat_aggregate_proj, s_src = X a_src) or read from s_src "
                         "(cogdl_gat_aggregate)")
    ap.add_argument("--counter-probe", metavar="JSON", default=None,
                    help="run one warmup step, one step and the calibration kernels between marker "
                         "kernels (for rocprofv3 --pmc), write the step's library launch names to JSON")
    ap.add_argument("--workloads-probe", metavar="JSON", default=None,
                    help="run each workloads-mode op once, cold, between marker kernels (for rocprofv3 "
                         "--pmc) and write the ops' keys to JSON")
    ap.add_argument("--wl-reps", type=int, default=5, help="timed calls per workload op in the default run")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-workload operator lines (workloads 1-4) of the default run")
    ap.add_argument("--no-live-counters", action="store_true",
                    help="do not run the counter probe under rocprofv3; take the HBM bytes from the "
                         "committed record under profiles/ when it matches the sources")
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                    help="FETCH_DIR WRITE_DIR PROBE_JSON [REQ_DIR]: write profiles/<workload>_hbm_traffic.json "
                         "and _hbm_counters.txt from a FETCH_SIZE and a WRITE_SIZE rocprofv3 run of "
                         "--counter-probe (and a run of the raw read-request counters), then exit")
    ap.add_argument("--summarize-workloads", nargs=3, metavar="PATH",
                    help="FETCH_DIR WRITE_DIR PROBE_JSON: write profiles/workloads_1_to_4_hbm_traffic.json "
                         "and _hbm_counters.txt from a FETCH_SIZE and a WRITE_SIZE rocprofv3 run of "
                         "--workloads-probe, then exit")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS_DIR", "COMMAND"),
                    help="write profiles/<workload>_kernel_stats.txt from the kernel statistics of a "
                         "rocprofv3 --kernel-trace --stats run (COMMAND: the command that made it), then exit")
    ap.add_argument("--summarize-plans", nargs=2, metavar=("SLICED_JSON", "PLAIN_JSON"),
                    help="write profiles/<workload>_sliced_vs_plain.txt from the JSON lines of a default "
                         "run and of a --plain-plans run (both with --no-cpu-baseline), then exit")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the steps, copy a buffer of this many MiB (counter calibration)")
    ap.add_argument("--workloads", action="store_true",
                    help="instead of the step: time each workload's own operators (workloads 1-4 "
                         "in their own dtypes), cold and warm, one JSON line per workload and op")
    ap.add_argument("--reps", type=int, default=20, help="--workloads: timed calls per op (cold and warm)")
    ap.add_argument("--warm-reps", type=int, default=3,
                    help="--workloads: untimed calls per op before timing (at least 1)")
    return ap.parse_args()


# ----------------------------------------------------------- byte models

def b_spmm(n_out, n_in, E, F, sx, sy):
    return 4 * (n_out + 1) + 8 * E + E * F * sx + n_out * F * sy


def b_csc(N, M, E):
    return 4 * (N + 1) + 8 * E + 4 * (M + 1) + 12 * E


def b_gat(N, E, H, D, sx, sy, alpha_out):
    return 4 * (N + 1) + 4 * E + 4 * N * H + 4 * E * H + E * H * D * sx + N * H * D * sy + (
        4 * E * H if alpha_out else 0)


def b_gat_proj(N, E, H, D, sx, sy):
    """The fused aggregation with source scores projected from the gathered rows: no score row
    per nonzero, the attention vector a_src (4HD) once instead."""
    return 4 * (N + 1) + 4 * E + 4 * N * H + E * H * D * sx + N * H * D * sy + 4 * H * D


def b_plan(N, n_units):
    return 4 * (N + 1) + 16 * n_units


# Compulsory bytes: every array once, the gathered feature rows (and GAT's
# per-source scores) read once each instead of once per nonzero.
def b_unique_spmm(n_out, n_in, E, F, sx, sy):
    return 4 * (n_out + 1) + 8 * E + n_in * F * sx + n_out * F * sy


def b_unique_gat(N, M, E, H, D, sx, sy):
    return 4 * (N + 1) + 4 * E + 4 * N * H + 4 * M * H + M * H * D * sx + N * H * D * sy


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# ----------------------------------------------------------- HBM counters
#
# The roofline fraction is taken from measured bytes: rocprofv3's FETCH_SIZE
# (bytes the L2 fetched from the fabric) and WRITE_SIZE (bytes it wrote) of the
# dominant kernel's dispatch in one step of the same workload, each scaled by
# what the counter reads for a copy of known size.  `--counter-probe` runs one
# warmup step, one step and the calibration kernels (libcogdl_calib.so: a
# copy, a streaming read, a gather of whole 128-byte lines and a gather of
# 16-byte rows, all of known traffic), each section between two marker
# kernels; bench.py runs it under rocprofv3 as a child process (one pass per
# counter) and reads the CSV back.  The calibrated record of such a run is
# also committed under profiles/ and used when the live run is unavailable
# and the library sources are unchanged.

MARKER = "bitwise_not"                     # the torch kernel launched between sections
PROBE_SECTIONS = ["step", "calib_copy", "calib_read", "calib_gather128", "calib_gather64", "calib_gather32",
                  "calib_gather16"]
GATHER_ROW_BYTES = (128, 64, 32, 16)
CALIB_BYTES = 1 << 30                      # copy and read size
CALIB_ROWS = 1 << 22                       # rows of each gather, distinct lines of a 2 GiB table
CALIB_TABLE_LINES = 1 << 24
HERE = os.path.dirname(os.path.abspath(__file__))


def calib_known_bytes():
    """(read, written) bytes of each calibration section, fixed by its arguments."""
    n = CALIB_ROWS
    out = {"calib_copy": (CALIB_BYTES, CALIB_BYTES), "calib_read": (CALIB_BYTES, 4096 * 4)}
    for rb in GATHER_ROW_BYTES:
        out[f"calib_gather{rb}"] = (n * rb + 4 * n, 4 * n)
    return out


def library_source_sha() -> str:
    """Hash of every library source and the header: a committed counter record holds
    only while it is unchanged."""
    import glob
    import hashlib
    csrc = os.path.join(HERE, "paper_2103_00959_amd", "csrc")
    files = sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.hpp")))
    files.append(os.path.join(HERE, "include", "cogdl.h"))
    return hashlib.sha256(b"".join(open(f, "rb").read() for f in files)).hexdigest()[:16]


def calib_lib():
    import ctypes
    L = ctypes.CDLL(os.path.join(HERE, "paper_2103_00959_amd", "libcogdl_calib.so"))
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.cogdl_calib_read.argtypes = [P, i64, P, P]
    L.cogdl_calib_copy.argtypes = [P, P, i64, P]
    L.cogdl_calib_gather.argtypes = [P, i64, i32, P, i64, P, P]
    return L


def read_dispatches(d: str, counter: str):
    """[(kernel name, counter value)] per dispatch, in dispatch order, from the CSV of a
    rocprofv3 --pmc <counter> --kernel-trace -d d -o run --output-format csv run."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise RuntimeError(f"no counter CSV under {d}")
    disp = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            k = (f, int(r["Dispatch_Id"]))
            e = disp.setdefault(k, [r["Kernel_Name"], 0.0])
            e[1] += float(r["Counter_Value"])
    return [tuple(v) for _, v in sorted(disp.items(), key=lambda kv: kv[0][1])]


def probe_sections(disp):
    """{section: [(name, value), ...]} between the marker dispatches of one probe run."""
    marks = [i for i, (n, _) in enumerate(disp) if MARKER in n]
    if len(marks) != len(PROBE_SECTIONS) + 1:
        raise RuntimeError(f"expected {len(PROBE_SECTIONS) + 1} marker dispatches, found {len(marks)}")
    return {sec: disp[marks[j] + 1:marks[j + 1]] for j, sec in enumerate(PROBE_SECTIONS)}


def summarize_probe(fetch_dir: str, write_dir: str, launches: list):
    """Calibrated HBM bytes of every dispatch of the probe's step (launch names from the
    library's trace, in order) and the calibration table."""
    F = probe_sections(read_dispatches(fetch_dir, "FETCH_SIZE"))
    W = probe_sections(read_dispatches(write_dir, "WRITE_SIZE"))
    known = calib_known_bytes()
    kib = 1024.0
    raw = {sec: (sum(v for _, v in F[sec]) * kib, sum(v for _, v in W[sec]) * kib) for sec in known}
    fetch_scale = known["calib_copy"][0] / raw["calib_copy"][0]
    write_scale = known["calib_copy"][1] / raw["calib_copy"][1]
    calib = {}
    for sec, (kr, kw) in known.items():
        fr, wr = raw[sec]
        calib[sec] = dict(known_read=kr, known_write=kw, fetch_raw=fr, write_raw=wr,
                          read_over_fetch_raw=kr / fr if fr else None,
                          fetch_calibrated_over_known=fr * fetch_scale / kr if kr else None)
    step_f, step_w = F["step"], W["step"]
    if len(step_f) != len(launches) or len(step_w) != len(launches):
        raise RuntimeError(f"step dispatches {len(step_f)}/{len(step_w)} != {len(launches)} library launches")
    step = [dict(launch=launches[i], kernel=step_f[i][0], fetch_bytes=step_f[i][1] * kib * fetch_scale,
                 write_bytes=step_w[i][1] * kib * write_scale) for i in range(len(launches))]
    return dict(fetch_scale=fetch_scale, write_scale=write_scale, calibration=calib, step=step,
                step_bytes=sum(d["fetch_bytes"] + d["write_bytes"] for d in step))


def kernel_traffic(summary, launch: str):
    """Calibrated bytes of the first dispatch of library launch `launch` in the step."""
    for d in summary["step"]:
        if d["launch"] == launch:
            return dict(bytes=d["fetch_bytes"] + d["write_bytes"], fetch_bytes=d["fetch_bytes"],
                        write_bytes=d["write_bytes"], kernel=d["kernel"])
    return None


def recorded_traffic(workload: str, profiles_dir: str | None = None):
    """The committed counter summary of the step (profiles/<workload>_hbm_traffic.json), or
    None when any library source changed since it was taken."""
    if profiles_dir is None:
        profiles_dir = os.path.join(HERE, "profiles")
    path = os.path.join(profiles_dir, f"{workload}_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_sha16") != library_source_sha():
        return None
    rec["source"] = os.path.relpath(path, HERE)
    return rec


def probe_command(args, out_json: str):
    cmd = [sys.executable, os.path.abspath(__file__), "--counter-probe", out_json, "--config", str(args.config),
           "--group-size", str(args.group_size)]
    if args.plain_plans:
        cmd.append("--plain-plans")
    if args.alpha_out:
        cmd.append("--alpha-out")
    cmd += ["--gat-scores", args.gat_scores]
    return cmd


def live_counters(args, timeout_s: float = 300.0):
    """Run the counter probe under rocprofv3 (a FETCH_SIZE pass, then a WRITE_SIZE pass) as
    child processes and summarize it; (summary, None) or (None, reason)."""
    import tempfile
    out_json = os.path.join(tempfile.mkdtemp(prefix="cogdl_probe_", dir="/tmp"), "probe.json")
    dirs, why = run_probe_passes(probe_command(args, out_json)[2:], out_json, timeout_s)
    if dirs is None:
        return None, why
    try:
        probe = json.load(open(out_json))
        summary = summarize_probe(dirs["fetch"], dirs["write"], probe["launches"])
    except Exception as e:       # noqa: BLE001  (a measurement aid: report, never fail the bench)
        return None, f"counter summary failed: {e}"
    summary["source"] = "live: rocprofv3 child runs of bench.py --counter-probe in this run"
    return summary, None


def cpu_baseline(g, X_bits, Xg_bits, sd, ss, H, D, F, budget_s, a_src=None):
    """Time the oracle (fp64, all host threads) on a random row sample of the
    SpMM and GAT steps, growing the sample until the budget is spent.  With
    a_src (projected source scores) the oracle first computes every node's
    source score (timed and counted: X read once), then aggregates."""
    import oracle
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    oracle.set_threads(threads)
    t_proj, b_proj = 0.0, 0
    if a_src is not None:
        t0 = time.perf_counter()
        ss64 = oracle.head_scores(Xg_bits, a_src, a_src, H, D, z_dtype=oracle.BF16)[0]
        t_proj = time.perf_counter() - t0
        ss = ss64.astype(np.float32)
        b_proj = g.n_cols * H * D * 2 + 4 * g.n_cols * H
    rng = np.random.default_rng(9)
    deg = np.diff(g.rowptr.astype(np.int64))
    rows_all = rng.permutation(g.n_rows).astype(np.int32)
    done_rows = 0
    t_total = 0.0
    bytes_total = 0
    edges_total = 0
    chunk = 2000
    while t_total < budget_s and done_rows < g.n_rows:
        sel = rows_all[done_rows:done_rows + chunk]
        done_rows += sel.size
        e = int(deg[sel].sum())
        t0 = time.perf_counter()
        oracle.spmm(g.rowptr, g.col, g.val, X_bits, x_dtype=oracle.BF16, rows=sel)
        oracle.gat(g.rowptr, g.col, sd, ss, Xg_bits, H, D, slope=0.2, x_dtype=oracle.BF16, rows=sel)
        t_total += time.perf_counter() - t0
        bytes_total += b_spmm(sel.size, g.n_cols, e, F, 2, 2) + (
            b_gat(sel.size, e, H, D, 2, 2, False) if a_src is None else b_gat_proj(sel.size, e, H, D, 2, 2))
        edges_total += 2 * e
        chunk = min(chunk * 2, 200000)
    t_total += t_proj
    bytes_total += b_proj
    return dict(value=bytes_total / t_total / 1e9, unit="GB/s", cores=threads, kind="oracle",
                cpu=cpu_model(),
                sample=(f"SpMM (F=256 bf16) + fused GAT (4x64 bf16) on {done_rows} random rows "
                        f"({edges_total // 2} nonzeros each) of the same graph, fp64 oracle"
                        + ("; the source scores of all nodes first (X a_src)" if a_src is not None else "")),
                seconds=t_total, edges_per_s=edges_total / t_total)


# ----------------------------------------------------------- main

def run_inference(cg, synth, dev, time_op_kernels, sliced=True):
    """End-to-end 2-layer GCN and GAT inference (hidden 128, GAT with 4 heads) on the
    Reddit-shaped graph: every step a library kernel, activations bf16."""
    import torch
    spec = synth.INFERENCE
    g = synth.config_graph(spec["graph"], verbose=True)
    N, E = g.n_rows, g.nnz
    k, hid, C, Hh, Dh = spec["F_in"], spec["hidden"], spec["classes"], spec["heads"], spec["head_dim"]
    rowptr = torch.from_numpy(g.rowptr).to(dev)
    col = torch.from_numpy(g.col).to(dev)
    val = torch.from_numpy(g.val).to(dev)

    def bf16(a):
        return torch.from_numpy(synth.f32_to_bf16_bits(a).view(np.int16)).to(dev).view(torch.bfloat16)

    X = bf16(synth.normal_f32((N, k), 7003))
    params = {}
    for kind in ("gcn", "gat"):
        p = synth.model_params(kind, k, hid, C, Hh, seed=7100 if kind == "gcn" else 7200)
        params[kind] = {n: (bf16(v) if n.startswith("W") else torch.from_numpy(v).to(dev))
                        for n, v in p.items()}
    plan = cg.Plan(rowptr, E, max_feat=hid, max_heads=Hh, **(dict(col=col, n_cols=N) if sliced else {}))
    torch.cuda.synchronize()
    ms_gcn, k_gcn = time_op_kernels(lambda: cg.gcn_forward(rowptr, col, val, X, params["gcn"], plan=plan))
    ms_gat, k_gat = time_op_kernels(lambda: cg.gat_forward(rowptr, col, X, params["gat"], spec["slope"],
                                                           plan=plan))
    plan.close()
    lin = lambda n, kk, m: 2 * (n * kk + m * kk + n * m)                       # noqa: E731
    agg = lambda F: 4 * (N + 1) + 8 * E + E * F * 2 + N * F * 2                # noqa: E731
    gat_agg = lambda H, D: 4 * (N + 1) + 4 * E + 8 * N * H + 4 * E * H + E * H * D * 2 + N * H * D * 2  # noqa: E731
    b_gcn = lin(N, k, hid) + agg(hid) + lin(N, hid, C) + agg(C)
    b_gat = (lin(N, k, hid) + N * hid * 2 + 8 * N * Hh + gat_agg(Hh, Dh)
             + lin(N, hid, C) + N * C * 2 + 8 * N + gat_agg(1, C))
    flops_dense = 2 * N * (k * hid + hid * C)
    log(f"inference on {spec['graph']}: GCN {ms_gcn:.3f} ms, GAT {ms_gat:.3f} ms")
    return {
        "workload": (f"{synth.CONFIGS[spec['graph']]['name']}: N={N}, nnz={E}, X bf16 N x {k}, "
                     f"hidden {hid}, {C} classes, GAT {Hh} heads x {Dh}; activations bf16, fp32 accumulation"),
        "gcn": dict(ms=ms_gcn, algorithmic_GB=b_gcn / 1e9, eff_GBps=b_gcn / (ms_gcn * 1e-3) / 1e9,
                    dense_TFLOPs=flops_dense / (ms_gcn * 1e-3) / 1e12, kernels_ms=k_gcn),
        "gat": dict(ms=ms_gat, algorithmic_GB=b_gat / 1e9, eff_GBps=b_gat / (ms_gat * 1e-3) / 1e9,
                    kernels_ms=k_gat),
        "paper_context": "2-layer GCN / GAT inference on Reddit (232,965 nodes, 11.6M edges): "
                         "0.022 s / 0.080 s on an RTX 3090 with CogDL; this graph has 114.6M edges",
    }


# Library sources behind the operators of the workloads mode (balancer, scan and radix
# sort, transpose, SpMM, edge softmax and GAT aggregation).
WORKLOAD_SOURCES = ["common.hpp", "internal.hpp", "primitives.hip", "plan.hip", "csc.hip",
                    "spmm_kernel.hpp", "spmm.hip", "gat_kernel.hpp", "gat.hip"]


def workloads_source_sha() -> str:
    """Hash of the sources of the workloads mode's operators and the header: the workload
    counters recorded under profiles/ hold only while it is unchanged."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    csrc = os.path.join(here, "paper_2103_00959_amd", "csrc")
    files = [os.path.join(csrc, f) for f in WORKLOAD_SOURCES] + [os.path.join(here, "include", "cogdl.h")]
    return hashlib.sha256(b"".join(open(f, "rb").read() for f in files)).hexdigest()[:16]


def recorded_workload_traffic(profiles_dir: str | None = None):
    """{"<workload>/<op>": {fetch_bytes, write_bytes, l2_hit, ...}} from the committed
    rocprofv3 summary of a --workloads run (HBM bytes of one cold call of each op), or
    None when any library source changed since the counters were taken."""
    if profiles_dir is None:
        profiles_dir = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles")
    path = os.path.join(profiles_dir, "workloads_1_to_4_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_sha16") != workloads_source_sha():
        return None
    return rec.get("ops")


def oracle_rate(run, units, budget_s, chunk=256, full=False):
    """Time the oracle over a random sample of `units` output rows (or columns), growing
    the chunk until `budget_s` is spent or every unit is done; run(sel) does one chunk
    and returns (algorithmic bytes, nonzeros) of it.  full: one call over all units."""
    if full:
        t0 = time.perf_counter()
        b, e = run(None)
        return dict(seconds=time.perf_counter() - t0, bytes=b, edges=e, units=units)
    order = np.random.default_rng(11).permutation(units).astype(np.int32)
    done, t, b_tot, e_tot = 0, 0.0, 0, 0
    while done < units and (done == 0 or t < budget_s):
        sel = np.sort(order[done:done + chunk])
        done += sel.size
        t0 = time.perf_counter()
        b, e = run(sel)
        t += time.perf_counter() - t0
        b_tot += b
        e_tot += e
        chunk = min(chunk * 2, 1 << 18)
    return dict(seconds=t, bytes=b_tot, edges=e_tot, units=done)


def run_workloads(reps=20, warm_reps=3, cpu=True, cpu_budget_s=2.0, hbm=None, probe=None, emit=None):
    """Each workload's operators in its own configuration (fp32 features; column-sliced plans
    on AUTO with the default group size), one JSON line per (workload, op).  Cold: a 1 GiB buffer is
    written before every timed call, so L2 and the Infinity Cache hold none of its inputs;
    warm: the same call back to back.  Median and minimum of `reps` calls after `warm_reps`
    untimed ones; plan creation and the transpose are preprocessing, reported on their own.
    Each line also carries the compulsory-byte rate, GFLOP/s, whether the gathered table fits
    the 256 MB Infinity Cache, a 1 GiB copy's rate (the achievable ceiling), the HBM bytes
    of one cold call from the committed rocprofv3 counters of this mode (when the library
    sources are unchanged since), and the fp64 CPU oracle's rate on the same op (all host
    threads; also one thread for workloads 1 and 2, whose ops the oracle does whole).

    hbm: {"<workload>/<op>": {fetch_bytes, write_bytes}} measured in this run (else the
    committed record is used).  probe: a path; instead of timing, every op runs once, cold
    (after the 1 GiB flush), between two marker kernels, and the ops' keys go to that JSON
    file (run under rocprofv3 for the counters).  emit: called with each record (default:
    print it as a JSON line).  Returns the records."""
    import torch

    import paper_2103_00959_amd as cg
    from paper_2103_00959_amd import synth

    dev = torch.device("cuda:0")
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    # a dispatch of a kernel no op uses opens and closes each op's section of a kernel trace
    marker = torch.zeros(1, dtype=torch.int32, device=dev)

    # achievable ceiling (and the counters' calibration): a plain 1 GiB device copy
    cp_dst = torch.empty_like(flush)
    flush.fill_(3)
    cp_ms = []
    for _ in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        cp_dst.copy_(flush)
        e1.record()
        torch.cuda.synchronize()
        cp_ms.append(e0.elapsed_time(e1))
    copy_GBps = 2 * (1 << 30) / (float(np.median(cp_ms[1:])) * 1e-3) / 1e9
    del cp_dst
    log(f"1 GiB copy: {copy_GBps:.0f} GB/s")
    hbm_source = "live" if hbm is not None else "profiles/workloads_1_to_4_hbm_traffic.json"
    if hbm is None:
        hbm = recorded_workload_traffic()
    records, probe_keys = [], []
    if emit is None:
        emit = lambda r: print(json.dumps(r), flush=True)          # noqa: E731
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    cpu_name = cpu_model()
    if cpu:
        import oracle

    def times(fn):
        if probe:
            fn()                             # warm (plans, caches of first use)
            flush.fill_(1)
            torch.cuda.synchronize()
            marker.bitwise_not_()
            fn()
            marker.bitwise_not_()
            torch.cuda.synchronize()
            return None
        # the first untimed call is traced to count the library launches of one call
        marker.bitwise_not_()
        cg.trace_enable(256)
        cg.trace_reset()
        fn()
        torch.cuda.synchronize()
        launches = len(cg.trace_read())
        cg.trace_enable(0)
        for _ in range(max(warm_reps, 1) - 1):
            fn()
        cold, warm = [], []
        for _ in range(reps):
            flush.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            cold.append(e0.elapsed_time(e1))
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        evs[0].record()
        for i in range(reps):
            fn()
            evs[i + 1].record()
        torch.cuda.synchronize()
        warm = [evs[i].elapsed_time(evs[i + 1]) for i in range(reps)]
        marker.bitwise_not_()           # and closes it
        return cold, warm, launches

    def oracle_line(k, run, units, whole=False, parallel=True):
        """CPU oracle timing of one op: all threads on a bounded random sample of the output
        rows (the whole op for workloads 1 and 2, and always when whole = True), plus one
        thread over the whole op for workloads 1 and 2.  parallel = False: that oracle
        routine is a serial loop, so one thread is what it uses."""
        if not cpu:
            return None
        oracle.set_threads(threads)
        r = oracle_rate(run, units, cpu_budget_s, full=whole or k <= 2)
        out = dict(kind="oracle", cores=threads if parallel else 1, cpu=cpu_name, seconds=r["seconds"],
                   GBps=r["bytes"] / r["seconds"] / 1e9,
                   edges_per_s=r["edges"] / r["seconds"] if r["edges"] else None,
                   sample=("whole op" if r["units"] == units else f"{r['units']} of {units} random output rows"))
        if k <= 2 and parallel:
            oracle.set_threads(1)
            r1 = oracle_rate(run, units, cpu_budget_s, full=True)
            out.update(GBps_1core=r1["bytes"] / r1["seconds"] / 1e9, seconds_1core=r1["seconds"])
            oracle.set_threads(threads)
        return out

    def record(k, cfg, op, B, B_u, E, flop, table_bytes, res, cpu_rec):
        if probe:
            probe_keys.append(f"{cfg['name']}/{op}")
            return
        cold, warm, launches = res
        mc, mw = float(np.median(cold)), float(np.median(warm))
        out = {"workload": cfg["name"], "config": k, "op": op, "algorithmic_GB": B / 1e9,
               "unique_GB": B_u / 1e9,
               "cold_ms_median": mc, "cold_ms_min": min(cold),
               "warm_ms_median": mw, "warm_ms_min": min(warm),
               "cold_eff_GBps": B / (mc * 1e-3) / 1e9, "cold_pct_peak": B / (mc * 1e-3) / 1e9 / HBM_PEAK_GBPS,
               "warm_eff_GBps": B / (mw * 1e-3) / 1e9,
               "cold_unique_GBps": B_u / (mc * 1e-3) / 1e9,
               "cold_edges_per_s": E / (mc * 1e-3) if E else None,
               "cold_GFLOPps": flop / (mc * 1e-3) / 1e9 if flop else None,
               "cache_resident": (table_bytes <= (256 << 20)) if table_bytes else None,
               "copy_GBps": copy_GBps, "launches_per_call": launches, "plans": "column-sliced",
               "hbm_GBps": None, "l2_hit": None, "hbm_source": None, "cpu_oracle": cpu_rec}
        h = hbm.get(f"{cfg['name']}/{op}") if hbm else None
        if h:
            out["hbm_GB"] = (h["fetch_bytes"] + h["write_bytes"]) / 1e9
            out["hbm_GBps"] = (h["fetch_bytes"] + h["write_bytes"]) / (mc * 1e-3) / 1e9
            out["hbm_frac"] = out["hbm_GBps"] / HBM_PEAK_GBPS
            out["l2_hit"] = h.get("l2_hit")
            out["hbm_source"] = hbm_source
        records.append(out)
        emit(out)
        log(f"{cfg['name']} {op}: cold {mc:.3f} ms ({out['cold_pct_peak'] * 100:.1f}% of peak), "
            f"warm {mw:.3f} ms" + (f", oracle {cpu_rec['GBps']:.2f} GB/s" if cpu_rec else ""))

    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)   # noqa: E731
    for k in (1, 2, 3, 4):
        cfg = synth.CONFIGS[k]
        g = synth.config_graph(k, verbose=True)
        N, M, E = g.n_rows, g.n_cols, g.nnz
        deg = np.diff(g.rowptr.astype(np.int64))
        rowptr, col = up(g.rowptr), up(g.col)
        val = up(g.val) if g.val is not None else None
        t0 = time.perf_counter()
        plan = cg.Plan(rowptr, E, max_feat=max(cfg.get("F", 1), cfg.get("H", 1) * cfg.get("D", 1)),
                       max_heads=cfg.get("H", 0), col=col, n_cols=M)
        torch.cuda.synchronize()
        log(f"{cfg['name']}: plan created in {(time.perf_counter() - t0) * 1e3:.1f} ms (host clock)")
        res = times(lambda: plan.rebuild(rowptr))
        inf = plan.info()
        Bp = b_plan(N, inf["n_units"])

        def run_plan(sel):
            oracle.neighbor_groups(g.rowptr, inf["group_size"], inf["mode"])
            return Bp, 0
        record(k, cfg, "plan_rebuild", Bp, Bp, 0, 0, 0, res, oracle_line(k, run_plan, N, True, False))
        if "F" in cfg:
            F = cfg["F"]
            Xn = synth.normal_f32((M, F), 2000 + k)
            X = up(Xn)
            Y = torch.empty((N, F), dtype=torch.float32, device=dev)
            res = times(lambda: cg.spmm(rowptr, col, val, X, plan=plan, out=Y))

            def run_spmm(sel):
                oracle.spmm(g.rowptr, g.col, g.val, Xn, rows=sel)
                n, e = (N, E) if sel is None else (sel.size, int(deg[sel].sum()))
                return b_spmm(n, M, e, F, 4, 4), e
            record(k, cfg, "spmm", b_spmm(N, M, E, F, 4, 4), b_unique_spmm(N, M, E, F, 4, 4), E,
                   2 * E * F, M * F * 4, res, oracle_line(k, run_spmm, N))
            if k == 2:
                colptr, row_t, val_t, perm = cg.csr_to_csc(rowptr, col, val, M)
                ws = torch.empty(cg.csr_to_csc_workspace(N, M, E), dtype=torch.uint8, device=dev)
                res = times(lambda: cg.csr_to_csc(rowptr, col, val, M, workspace=ws))

                def run_csc(sel):
                    oracle.csr_to_csc(g.rowptr, g.col, g.val, M)
                    return b_csc(N, M, E), E
                record(k, cfg, "csr_to_csc", b_csc(N, M, E), b_csc(N, M, E), E, 0, 0, res,
                       oracle_line(k, run_csc, M, True, False))
                plan_t = cg.Plan(colptr, E, max_feat=F, col=row_t, n_cols=N)
                Gn = synth.normal_f32((N, F), 4000 + k)
                G = up(Gn)
                dX = torch.empty((M, F), dtype=torch.float32, device=dev)
                res = times(lambda: cg.spmm_t(colptr, row_t, val_t, G, plan_t=plan_t, out=dX))
                cdeg = np.bincount(g.col, minlength=M).astype(np.int64)

                def run_spmm_t(sel):
                    oracle.spmm_t(g.rowptr, g.col, g.val, Gn, M, cols=sel)
                    n, e = (M, E) if sel is None else (sel.size, int(cdeg[sel].sum()))
                    return b_spmm(n, N, e, F, 4, 4), e
                record(k, cfg, "spmm_t", b_spmm(M, N, E, F, 4, 4), b_unique_spmm(M, N, E, F, 4, 4), E,
                       2 * E * F, N * F * 4, res, oracle_line(k, run_spmm_t, M, True, False))
                plan_t.close()
                del colptr, row_t, val_t, perm, ws, G, dX
            del X, Y
        if "H" in cfg:
            H, D = cfg["H"], cfg["D"]
            rng = np.random.default_rng(3000 + k)
            sd_n = rng.standard_normal((N, H), dtype=np.float32)
            ss_n = rng.standard_normal((M, H), dtype=np.float32)
            Xg_n = synth.normal_f32((M, H * D), 2100 + k)
            s_dst, s_src = up(sd_n), up(ss_n)
            Xg = up(Xg_n).view(M, H, D)
            Yg = torch.empty((N, H, D), dtype=torch.float32, device=dev)
            alpha = torch.empty((E, H), dtype=torch.float32, device=dev)
            res = times(lambda: cg.sddmm_edge_softmax(rowptr, col, s_dst, s_src, 0.2, plan=plan, out=alpha))
            b_sm = lambda n, e: 4 * (n + 1) + 4 * e + 4 * n * H + 4 * e * H + 4 * e * H   # noqa: E731

            def run_softmax(sel):
                oracle.edge_softmax(g.rowptr, g.col, sd_n, ss_n, slope=0.2, rows=sel)
                n, e = (N, E) if sel is None else (sel.size, int(deg[sel].sum()))
                return b_sm(n, e), e
            record(k, cfg, "sddmm_edge_softmax", b_sm(N, E), b_sm(N, E) - 4 * E * H + 4 * M * H, E,
                   0, M * H * 4, res, oracle_line(k, run_softmax, N))
            for a_out in (False, True):
                res = times(lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan,
                                                     out=Yg, alpha_out=alpha if a_out else None))

                def run_gat(sel, a_out=a_out):
                    oracle.gat(g.rowptr, g.col, sd_n, ss_n, Xg_n, H, D, slope=0.2, rows=sel)
                    n, e = (N, E) if sel is None else (sel.size, int(deg[sel].sum()))
                    return b_gat(n, e, H, D, 4, 4, a_out), e
                record(k, cfg, "gat_aggregate" + ("_alpha_out" if a_out else ""),
                       b_gat(N, E, H, D, 4, 4, a_out),
                       b_unique_gat(N, M, E, H, D, 4, 4) + (4 * E * H if a_out else 0), E,
                       2 * E * H * D + 8 * E * H, M * H * D * 4, res, oracle_line(k, run_gat, N))
            del s_dst, s_src, Xg, Yg, alpha
        plan.close()
        del rowptr, col, val
        torch.cuda.empty_cache()
    if probe:
        # the copy of known size that scales the counters, as its own section
        import ctypes
        C = calib_lib()
        dst = torch.empty_like(flush)
        torch.cuda.synchronize()
        marker.bitwise_not_()
        rc = C.cogdl_calib_copy(ctypes.c_void_p(flush.data_ptr()), ctypes.c_void_p(dst.data_ptr()), CALIB_BYTES,
                                cg._stream())
        marker.bitwise_not_()
        torch.cuda.synchronize()
        if rc:
            raise SystemExit("calibration copy refused its arguments")
        probe_keys.append("calib_copy")
        with open(probe, "w") as f:
            json.dump({"keys": probe_keys}, f)
        log(f"workloads probe done: {len(probe_keys)} sections")
    return records


def summarize_workloads_probe(fetch_dir: str, write_dir: str, keys: list):
    """{"<workload>/<op>": {fetch_bytes, write_bytes}} of one cold call of each op of a
    --workloads-probe run: the dispatches between each pair of markers, scaled by what the
    counters read for the closing 1 GiB copy."""
    out = {}
    for counter, d, field in (("FETCH_SIZE", fetch_dir, "fetch_bytes"), ("WRITE_SIZE", write_dir, "write_bytes")):
        disp = read_dispatches(d, counter)
        marks = [i for i, (n, _) in enumerate(disp) if MARKER in n]
        if len(marks) != 2 * len(keys):
            raise RuntimeError(f"expected {2 * len(keys)} marker dispatches, found {len(marks)}")
        sums = [sum(v for _, v in disp[marks[2 * i] + 1:marks[2 * i + 1]]) * 1024.0 for i in range(len(keys))]
        scale = CALIB_BYTES / sums[keys.index("calib_copy")]
        for key, b in zip(keys, sums):
            out.setdefault(key, {})[field] = b * scale
            out[key][field.replace("bytes", "scale")] = scale
    out.pop("calib_copy")
    return out


def run_probe_passes(probe_args: list, out_json: str, timeout_s: float = 300.0):
    """Run `bench.py <probe_args>` under rocprofv3, one FETCH_SIZE and one WRITE_SIZE pass,
    as child processes; ({"fetch": dir, "write": dir}, None) or (None, reason)."""
    import shutil
    import signal
    import subprocess
    import tempfile
    exe = shutil.which("rocprofv3") or "/opt/rocm/bin/rocprofv3"
    if not os.path.exists(exe):
        return None, "rocprofv3 not found"
    base = tempfile.mkdtemp(prefix="cogdl_counters_", dir="/tmp")
    env = dict(os.environ, TMPDIR="/tmp")
    dirs = {}
    for tag, ctr in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        d = os.path.join(base, tag)
        cmd = [exe, "--pmc", ctr, "--kernel-trace", "-d", d, "-o", "run", "--output-format", "csv", "--",
               sys.executable, os.path.abspath(__file__)] + probe_args
        log(f"counters: {ctr} pass of {' '.join(probe_args[:1])}")
        with open(os.path.join(base, f"{tag}.log"), "w") as lf:
            p = subprocess.Popen(cmd, cwd="/tmp", env=env, stdout=lf, stderr=subprocess.STDOUT,
                                 start_new_session=True)
            try:
                rc = p.wait(timeout=timeout_s)
            except subprocess.TimeoutExpired:
                os.killpg(p.pid, signal.SIGKILL)
                p.wait()
                return None, f"{ctr} pass timed out after {timeout_s:.0f} s"
        # rocprofv3 may end with a segmentation fault after the program finished and
        # its results are complete: the probe's own output file says whether it did
        if rc != 0 and not os.path.exists(out_json):
            return None, f"{ctr} pass exited with {rc}"
        dirs[tag] = d
    return dirs, None


def live_workload_counters(args, timeout_s: float = 300.0):
    """Counter bytes of one cold call of every workloads-mode op, measured in this run."""
    import tempfile
    out_json = os.path.join(tempfile.mkdtemp(prefix="cogdl_wlprobe_", dir="/tmp"), "probe.json")
    dirs, why = run_probe_passes(["--workloads-probe", out_json], out_json, timeout_s)
    if dirs is None:
        return None, why
    try:
        return summarize_workloads_probe(dirs["fetch"], dirs["write"], json.load(open(out_json))["keys"]), None
    except Exception as e:       # noqa: BLE001  (a measurement aid: report, never fail the bench)
        return None, f"workload counter summary failed: {e}"


def counter_probe(args, cg, step, dev):
    """The probe run under rocprofv3: one warmup step, then [marker] one step [marker] and the
    calibration kernels, each followed by a marker; the step's library launch names go to
    args.counter_probe (JSON), so that its dispatches can be named one by one."""
    import ctypes

    import torch
    # calibration inputs first: every kernel that prepares them runs before the first marker
    C = calib_lib()
    s = cg._stream()
    P = lambda t: ctypes.c_void_p(t.data_ptr())                      # noqa: E731
    src = torch.full((CALIB_BYTES,), 1, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    sink = torch.empty(4096, dtype=torch.int32, device=dev)
    table = torch.full((CALIB_TABLE_LINES * 128,), 2, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device=dev).manual_seed(17)
    perm = torch.randperm(CALIB_TABLE_LINES, generator=gen, device=dev, dtype=torch.int64)
    # each gather reads its own rows: CALIB_ROWS distinct lines, disjoint between sections
    idx = [perm[i * CALIB_ROWS:(i + 1) * CALIB_ROWS].to(torch.int32).contiguous()
           for i in range(len(GATHER_ROW_BYTES))]
    lo, hi = int(perm.min()), int(perm.max())
    assert 0 <= lo and hi < CALIB_TABLE_LINES        # every gathered row is inside the table
    out = torch.empty(CALIB_ROWS, dtype=torch.int32, device=dev)
    marker = torch.zeros(1, dtype=torch.int32, device=dev)
    step()
    torch.cuda.synchronize()
    cg.trace_enable(4096)
    cg.trace_filter(None)
    cg.trace_reset()
    marker.bitwise_not_()
    step()
    marker.bitwise_not_()
    torch.cuda.synchronize()
    launches = [n for n, _ in cg.trace_read()]
    cg.trace_enable(0)
    checks = [C.cogdl_calib_copy(P(src), P(dst), CALIB_BYTES, s)]
    marker.bitwise_not_()
    checks.append(C.cogdl_calib_read(P(src), CALIB_BYTES, P(sink), s))
    marker.bitwise_not_()
    for rb, ix in zip(GATHER_ROW_BYTES, idx):
        checks.append(C.cogdl_calib_gather(P(table), 128, rb, P(ix), CALIB_ROWS, P(out), s))
        marker.bitwise_not_()
    torch.cuda.synchronize()
    if any(checks):
        raise SystemExit(f"calibration kernel refused its arguments: {checks}")
    with open(args.counter_probe, "w") as f:
        json.dump({"launches": launches, "sections": PROBE_SECTIONS}, f)
    log(f"counter probe done: {len(launches)} library launches in the step")


REQ_COUNTERS = ("TCC_BUBBLE_sum", "TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum")


def request_mix(req_dir, launches):
    """Read requests the L2 sent to the fabric per section (and per step launch), by size:
    128-byte (TCC_BUBBLE), 32-byte (TCC_EA0_RDREQ_32B) and the 64-byte rest of TCC_EA0_RDREQ
    (the counters FETCH_SIZE is computed from)."""
    secs = {c: probe_sections(read_dispatches(req_dir, c)) for c in REQ_COUNTERS}
    out = {}
    for sec in PROBE_SECTIONS:
        rows = list(zip(*(secs[c][sec] for c in REQ_COUNTERS)))
        names = ["calib"] if sec != "step" else launches
        if sec == "step" and len(rows) != len(launches):
            raise RuntimeError("request-counter run does not match the probe's launches")
        for i, r in enumerate(rows):
            b128, tot, b32 = (v for _, v in r)
            key = sec if sec != "step" else f"step/{i:02d} {names[i]}"
            if sec != "step" and i > 0:
                prev = out[key]
                b128, tot, b32 = prev["req128"] + b128, prev["req_total"] + tot, prev["req32"] + b32
            out[key] = dict(req128=b128, req32=b32, req64=tot - b128 - b32, req_total=tot)
    return out


def write_counter_profile(args, fetch_dir, write_dir, probe_json, req_dir=None):
    """profiles/<workload>_hbm_traffic.json (the record bench.py falls back on) and a readable
    _hbm_counters.txt from one FETCH_SIZE and one WRITE_SIZE run of --counter-probe."""
    from paper_2103_00959_amd import synth
    cfg = synth.CONFIGS[args.config]
    probe = json.load(open(probe_json))
    summ = summarize_probe(fetch_dir, write_dir, probe["launches"])
    summ["source_sha16"] = library_source_sha()
    summ["workload"] = cfg["name"]
    flags = " ".join(probe_command(args, "PROBE_JSON")[4:])
    cmd = ("cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --kernel-trace -d DIR -o run --output-format csv -- "
           f"python3 bench.py --counter-probe PROBE_JSON {flags}")
    summ["commands"] = {"fetch": cmd.format(c="FETCH_SIZE"), "write": cmd.format(c="WRITE_SIZE")}
    out = os.path.join(HERE, "profiles", f"{cfg['name']}_hbm_traffic.json")
    json.dump(summ, open(out, "w"), indent=1)
    lines = [f"# HBM bytes of one step of {cfg['name']} on one MI355X, per dispatch, from rocprofv3 counters",
             f"# FETCH_SIZE: {summ['commands']['fetch']}",
             f"# WRITE_SIZE: {summ['commands']['write']}",
             f"# (bench.py runs the same two passes itself unless --no-live-counters; this record is its fallback)",
             f"# library sources sha256[:16] {summ['source_sha16']}",
             "# calibration (kernels of known traffic, libcogdl_calib.so): bytes the section must read / write,",
             "# raw counter bytes, and known / raw; the copy's ratios are the scales applied to every dispatch",
             f"# {'section':18s} {'known_read':>12s} {'fetch_raw':>12s} {'read/raw':>9s} {'known_wr':>12s} "
             f"{'write_raw':>12s} {'wr/raw':>7s}"]
    for sec, c in summ["calibration"].items():
        lines.append(f"# {sec:18s} {c['known_read']:12.4e} {c['fetch_raw']:12.4e} "
                     f"{c['known_read'] / c['fetch_raw']:9.4f} {c['known_write']:12.4e} {c['write_raw']:12.4e} "
                     f"{(c['known_write'] / c['write_raw']) if c['write_raw'] else float('nan'):7.4f}")
    lines.append(f"# scales: fetch x{summ['fetch_scale']:.4f}, write x{summ['write_scale']:.4f}")
    lines.append(f"{'launch':22s} {'kernel':64s} {'fetch_GB':>9s} {'write_GB':>9s}")
    for d in summ["step"]:
        lines.append(f"{d['launch']:22s} {d['kernel'][:64]:64s} {d['fetch_bytes'] / 1e9:9.4f} "
                     f"{d['write_bytes'] / 1e9:9.4f}")
    lines.append(f"step total {summ['step_bytes'] / 1e9:.3f} GB")
    if req_dir:
        mix = request_mix(req_dir, probe["launches"])
        summ["read_requests"] = mix
        json.dump(summ, open(out, "w"), indent=1)
        lines.append("# read requests the L2 sent to the fabric, by size (raw counts: "
                     + " ".join(REQ_COUNTERS) + f"), command: {cmd.format(c=' '.join(REQ_COUNTERS))}")
        lines.append(f"{'section / launch':40s} {'128B':>12s} {'64B':>12s} {'32B':>12s} {'bytes_by_size':>14s}")
        for k, v in mix.items():
            if k.startswith("step/") and not any(t in k for t in (" spmm", " gat", "radix_scatter")):
                continue
            by = 128 * v["req128"] + 64 * v["req64"] + 32 * v["req32"]
            lines.append(f"{k:40s} {v['req128']:12.4e} {v['req64']:12.4e} {v['req32']:12.4e} {by:14.4e}")
    open(os.path.join(HERE, "profiles", f"{cfg['name']}_hbm_counters.txt"), "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def write_workload_profile(fetch_dir, write_dir, probe_json, out_dir=None):
    """profiles/workloads_1_to_4_hbm_traffic.json (the record the workload lines fall back on)
    and a readable .txt from one FETCH_SIZE and one WRITE_SIZE run of --workloads-probe."""
    keys = json.load(open(probe_json))["keys"]
    ops = summarize_workloads_probe(fetch_dir, write_dir, keys)
    cmd = ("cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --kernel-trace -d DIR -o run --output-format csv -- "
           "python3 bench.py --workloads-probe PROBE_JSON")
    rec = {"source_sha16": workloads_source_sha(), "ops": ops,
           "commands": {"fetch": cmd.format(c="FETCH_SIZE"), "write": cmd.format(c="WRITE_SIZE"),
                        "summary": "python3 bench.py --summarize-workloads FETCH_DIR WRITE_DIR PROBE_JSON"}}
    base = os.path.join(out_dir or os.path.join(HERE, "profiles"), "workloads_1_to_4_hbm")
    json.dump(rec, open(base + "_traffic.json", "w"), indent=1)
    lines = ["# HBM bytes of one cold call of each workloads-mode operator (workloads 1-4, their own dtypes),",
             "# one MI355X: the dispatches between the op's two marker kernels, each counter scaled by what it",
             "# reads for the run's closing plain 1 GiB device copy",
             f"# FETCH_SIZE: {rec['commands']['fetch']}",
             f"# WRITE_SIZE: {rec['commands']['write']}",
             f"# summary: {rec['commands']['summary']}",
             f"# workload-op sources sha256[:16] {rec['source_sha16']} (the record is ignored once they change)",
             f"{'workload/op':48s} {'fetch_GB':>9s} {'write_GB':>9s} {'fetch_x':>8s} {'write_x':>8s}"]
    for k, v in ops.items():
        lines.append(f"{k:48s} {v['fetch_bytes'] / 1e9:9.4f} {v['write_bytes'] / 1e9:9.4f} "
                     f"{v['fetch_scale']:8.3f} {v['write_scale']:8.3f}")
    open(base + "_counters.txt", "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def write_stats_profile(args, stats_dir, command, out_dir=None):
    """profiles/<workload>_kernel_stats.txt from run_kernel_stats.csv of a rocprofv3
    --kernel-trace --stats run: calls, average and total time per kernel."""
    import csv
    import glob
    from paper_2103_00959_amd import synth
    cfg = synth.CONFIGS[args.config]
    files = glob.glob(os.path.join(stats_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {stats_dir}")
    rows = list(csv.DictReader(open(files[0])))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = [f"# Kernel time of {cfg['name']}, one MI355X (rocprofv3 kernel statistics; durations in ms)",
             f"# command: {command}",
             f"# library sources sha256[:16] {library_source_sha()}",
             f"{'kernel':90s} {'calls':>6s} {'avg_ms':>9s} {'min_ms':>9s} {'max_ms':>9s} {'total_ms':>10s} {'pct':>6s}"]
    for r in rows:
        name = r["Name"].replace("cogdl::(anonymous namespace)::", "").replace("cogdl::", "")
        lines.append(f"{name[:90]:90s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e6:9.4f} "
                     f"{float(r['MinNs']) / 1e6:9.4f} {float(r['MaxNs']) / 1e6:9.4f} "
                     f"{float(r['TotalDurationNs']) / 1e6:10.3f} {float(r['Percentage']):6.2f}")
    out = os.path.join(out_dir or os.path.join(HERE, "profiles"), f"{cfg['name']}_kernel_stats.txt")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines[:30]))


def write_plans_profile(sliced_json, plain_json, out_dir=None):
    """profiles/<workload>_sliced_vs_plain.txt: the step, its operators and kernels, the operators
    outside the step and the inference workload side by side for the two kinds of balancer plan."""
    a, b = (json.loads(open(f).read().strip().splitlines()[-1]) for f in (sliced_json, plain_json))
    if a["config"]["workload"] != b["config"]["workload"]:
        raise SystemExit("the two runs measured different workloads")
    name = a["config"]["workload"].split(":")[0]
    rows = [("step ms (timed region)", a["ms_per_step"], b["ms_per_step"], 3),
            ("value GB/s (algorithmic)", a["value"], b["value"], 0)]
    rows += [(f"{k} ms", a["ops"][k]["ms"], b["ops"][k]["ms"], 3) for k in a["ops"] if k in b["ops"]]
    rows += [(f"kernel {k} ms", a["kernels"][k]["avg_ms"], b["kernels"][k]["avg_ms"], 3)
             for k in a["kernels"] if k in b["kernels"] and k.startswith(("spmm", "gat"))]
    oa, ob = a.get("ops_outside_step", {}), b.get("ops_outside_step", {})
    rows += [(f"outside the step: {k} ms", oa[k].get("ms"), ob[k].get("ms"), 3)
             for k in oa if k in ob and isinstance(oa[k], dict) and isinstance(ob[k], dict)]
    for m in ("gcn", "gat"):
        if m in a.get("inference", {}) and m in b.get("inference", {}):
            rows.append((f"inference {m.upper()} ms", a["inference"][m]["ms"], b["inference"][m]["ms"], 3))
    rows.append((f"roofline kernel avg ms ({a['roofline']['kernel']})", a["roofline"]["avg_ms"],
                 b["roofline"]["avg_ms"], 3))
    lines = [f"# Column-sliced vs plain balancer plans on {name}, one MI355X, same box, back to back",
             "# sliced: cd /tmp && python3 $GRAFT_REPO_ROOT/bench.py --no-cpu-baseline",
             "# plain:  cd /tmp && python3 $GRAFT_REPO_ROOT/bench.py --no-cpu-baseline --plain-plans",
             "# table:  python3 bench.py --summarize-plans SLICED_JSON PLAIN_JSON",
             f"# library sources sha256[:16] {library_source_sha()}",
             "# per-operator times: mean over the instrumented steps (events around every launch); step: "
             "the timed region; inference: the Reddit-shaped workload 3 graph with the same kind of plan",
             f"{'quantity':48s} {'sliced':>10s} {'plain':>10s}"]
    for label, x, y, nd in rows:
        if x is None or y is None:
            continue
        lines.append(f"{label:48s} {x:10.{nd}f} {y:10.{nd}f}")
    out = os.path.join(out_dir or os.path.join(HERE, "profiles"), f"{name}_sliced_vs_plain.txt")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path has no "
              f"multi-GPU mode in this build", file=sys.stderr)
        sys.exit(2)
    if args.workloads_probe:
        run_workloads(reps=1, warm_reps=1, cpu=False, probe=args.workloads_probe, emit=lambda r: None)
        return
    if args.workloads:
        wl_hbm = None
        if not args.no_live_counters:
            wl_hbm, why = live_workload_counters(args)
            if wl_hbm is None:
                log(f"live workload counters unavailable ({why})")
        run_workloads(reps=args.reps, warm_reps=args.warm_reps, cpu=not args.no_cpu_baseline, hbm=wl_hbm)
        return
    if args.summarize_workloads:
        write_workload_profile(*args.summarize_workloads)
        return
    if args.summarize_stats:
        write_stats_profile(args, *args.summarize_stats)
        return
    if args.summarize_plans:
        write_plans_profile(*args.summarize_plans)
        return
    if args.summarize_counters:
        if len(args.summarize_counters) not in (3, 4):
            raise SystemExit("--summarize-counters FETCH_DIR WRITE_DIR PROBE_JSON [REQ_DIR]")
        write_counter_profile(args, *args.summarize_counters)
        return
    import torch

    import paper_2103_00959_amd as cg
    from paper_2103_00959_amd import synth

    cfg = synth.CONFIGS[args.config]
    if "F" not in cfg or "H" not in cfg:
        raise SystemExit("the step needs a workload with both GCN (F) and GAT (H, D) features")
    log(f"workload {cfg['name']}; host threads {os.cpu_count()}")
    t0 = time.time()
    g = synth.config_graph(args.config, verbose=True)
    N, M, E = g.n_rows, g.n_cols, g.nnz
    F, H, D = cfg["F"], cfg["H"], cfg["D"]
    log(f"graph ready N={N} E={E} in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")

    def up(a, dt=None):
        t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return t.view(dt) if dt is not None else t

    rowptr, col, val = up(g.rowptr), up(g.col), up(g.val)
    if args.counter_probe:
        # The counter probe only measures memory traffic, which these kernels take from
        # the graph and the shapes alone (no access depends on a feature or score value):
        # normal features drawn on the device spare the host generation.
        gen = torch.Generator(device=dev).manual_seed(2000 + args.config)
        X = torch.randn((M, F), generator=gen, device=dev).to(torch.bfloat16)
        Gt = torch.randn((N, F), generator=gen, device=dev).to(torch.bfloat16)
        Xg = torch.randn((M, H, D), generator=gen, device=dev).to(torch.bfloat16)
        s_dst = torch.randn((N, H), generator=gen, device=dev)
        s_src = torch.randn((M, H), generator=gen, device=dev)
        a_src = torch.randn((H, D), generator=gen, device=dev) / float(np.sqrt(D))
    else:
        X32 = synth.normal_f32((M, F), 2000 + args.config)
        X_bits = synth.f32_to_bf16_bits(X32)
        del X32
        G_bits = synth.f32_to_bf16_bits(synth.normal_f32((N, F), 4000 + args.config))
        Xg_bits = synth.f32_to_bf16_bits(synth.normal_f32((M, H * D), 2100 + args.config))
        rng = np.random.default_rng(3000 + args.config)
        sd = rng.standard_normal((N, H), dtype=np.float32)
        ss = rng.standard_normal((M, H), dtype=np.float32)
        # the attention vector of the projected source scores: N(0, 1/D) per entry, so that
        # s_src = X a_src is N(0, 1) like the given scores
        a_src_h = (np.random.default_rng(3100 + args.config).standard_normal((H, D)) / np.sqrt(D)).astype(np.float32)
        X = up(X_bits.view(np.int16), torch.bfloat16)
        Gt = up(G_bits.view(np.int16), torch.bfloat16)
        Xg = up(Xg_bits.view(np.int16), torch.bfloat16).view(M, H, D)
        s_dst, s_src, a_src = up(sd), up(ss), up(a_src_h)
    log(f"features ready in {time.time() - t0:.1f}s")
    Y = torch.empty((N, F), dtype=torch.bfloat16, device=dev)
    dX = torch.empty((M, F), dtype=torch.bfloat16, device=dev)
    Yg = torch.empty((N, H, D), dtype=torch.bfloat16, device=dev)
    alpha = torch.empty((E, H), dtype=torch.float32, device=dev) if args.alpha_out else None
    colptr = torch.empty(M + 1, dtype=torch.int32, device=dev)
    row_t = torch.empty(E, dtype=torch.int32, device=dev)
    val_t = torch.empty(E, dtype=torch.float32, device=dev)
    perm = torch.empty(E, dtype=torch.int32, device=dev)
    ws = torch.empty(cg.csr_to_csc_workspace(N, M, E), dtype=torch.uint8, device=dev)
    L = cg.lib()
    stream = cg._stream

    def csc():
        cg._check(L.cogdl_csr_to_csc(N, M, E, cg._ptr(rowptr), cg._ptr(col), cg._ptr(val),
                                     cg._ptr(colptr), cg._ptr(row_t), cg._ptr(val_t), cg._ptr(perm),
                                     cg._ptr(ws), ws.numel(), stream()), "csr_to_csc")

    # column-sliced plans (each XCD gathers from its own eighth of the table), or plain ones
    sl = {} if args.plain_plans else dict(col=col, n_cols=M)
    sl_t = {} if args.plain_plans else dict(col=row_t, n_cols=N)
    plan = cg.Plan(rowptr, E, max_feat=max(F, H * D), max_heads=H, group_size=args.group_size, **sl)
    csc()
    plan_t = cg.Plan(colptr, E, max_feat=F, max_heads=H, group_size=args.group_size, **sl_t)
    torch.cuda.synchronize()
    info, info_t = plan.info(), plan_t.info()
    log(f"plan: {info['mode_name']} units={info['n_units']} long={info['n_long_units']} "
        f"split_rows={info['n_split_rows']} partials={info['n_partials']}; plan_t: "
        f"{info_t['mode_name']} units={info_t['n_units']} split_rows={info_t['n_split_rows']}")
    # Edges and directly written rows of the long-unit and tiny-unit kernels
    # (split rows are written by the reduce kernel): the algorithmic bytes of
    # an op are split exactly between its kernels.
    # A unit runs in the tiny-unit kernel when the plan uses neighbour groups larger than
    # the tiny size and the unit has at most that many edges (sliced plans keep one
    # long/tiny pair of ranges per XCD list, so the split is by size, not by position).
    TINY = 8                                                        # kTinyUnit
    def unit_split(p, inf):
        un = p.units().cpu().numpy().astype(np.int64)
        size = un[:, 2] - un[:, 1]
        direct = un[:, 3] < 0
        tiny = (size <= TINY) if (inf["mode"] == 2 and inf["group_size"] > TINY) else np.zeros(len(un), bool)
        assert int((~tiny).sum()) == inf["n_long_units"]
        return dict(E_long=int(size[~tiny].sum()), R_long=int((direct & ~tiny).sum()),
                    E_tiny=int(size[tiny].sum()), R_tiny=int((direct & tiny).sum()),
                    R_split=inf["n_split_rows"])
    us, us_t = unit_split(plan, info), unit_split(plan_t, info_t)

    OPS = ["plan", "spmm", "csr_to_csc", "plan_t", "spmm_t", "gat_aggregate"]
    proj = args.gat_scores == "proj" and not args.alpha_out
    gat_k = "gat_proj" if proj else "gat"          # the GAT step's long-unit kernel

    def step(evs=None):
        mark = (lambda i: evs[i].record()) if evs is not None else (lambda i: None)
        mark(0)
        plan.rebuild(rowptr)                                                   # a1
        mark(1)
        cg.spmm(rowptr, col, val, X, plan=plan, out=Y)                         # a2
        mark(2)
        csc()                                                                  # a3
        mark(3)
        plan_t.rebuild(colptr)                                                 # a1 (CSC)
        mark(4)
        cg.spmm_t(colptr, row_t, val_t, Gt, plan_t=plan_t, out=dX)             # a4
        mark(5)
        if proj:                                                               # a5-a7
            cg.gat_aggregate_proj(rowptr, col, s_dst, a_src, Xg, 0.2, plan=plan, out=Yg)
        else:
            cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan, out=Yg, alpha_out=alpha)
        mark(6)

    if args.counter_probe:
        counter_probe(args, cg, step, dev)
        return

    if args.calib_copy_mib > 0:
        # a plain device-to-device copy of known size, for scaling the HBM counters
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mib} MiB done")
        del src, dst

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup {i + 1}/{args.warmup} done")

    # Timed region: the K steps with HIP events only around the launches of
    # the roofline candidates (an event pair costs the stream a few
    # microseconds; around every launch they would add about 0.6 ms a step).
    ROOF = ("spmm", "spmm_t", gat_k)
    cg.trace_enable(128 * args.steps + 64)
    cg.trace_filter(ROOF)
    cg.trace_reset()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    ev0.record()
    for i in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = ev0.elapsed_time(ev1) / args.steps
    roof_trace = cg.trace_read()
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step (wall {t_wall:.2f}s)")

    # Instrumented pass (after the timed region, not part of it): K more steps
    # with events between operators and around every library launch, for the
    # per-operator and per-kernel breakdown.
    cg.trace_filter(None)
    cg.trace_reset()
    step_evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(OPS) + 1)]
                for _ in range(args.steps)]
    for i in range(args.steps):
        step(step_evs[i])
    torch.cuda.synchronize()
    op_all = {op: [e[j].elapsed_time(e[j + 1]) for e in step_evs] for j, op in enumerate(OPS)}
    op_ms = {op: sum(v) / args.steps for op, v in op_all.items()}
    ms_step_instr = sum(e[0].elapsed_time(e[-1]) for e in step_evs) / args.steps
    trace = cg.trace_read()
    cg.trace_enable(0)
    cg.trace_filter(None)
    log(f"instrumented pass: {ms_step_instr:.3f} ms/step")

    # per-kernel device time from the library's own HIP events
    per = {}
    for name, ms in trace:
        s = per.setdefault(name, [0.0, 0])
        s[0] += ms
        s[1] += 1
    kernels = {k: dict(total_ms=v[0] / args.steps, launches=v[1] // args.steps,
                       avg_ms=v[0] / v[1]) for k, v in per.items()}

    B = {
        "plan": b_plan(N, info["n_units"]),
        "plan_t": b_plan(M, info_t["n_units"]),
        "spmm": b_spmm(N, M, E, F, 2, 2),
        "csr_to_csc": b_csc(N, M, E),
        "spmm_t": b_spmm(M, N, E, F, 2, 2),
        "gat_aggregate": b_gat_proj(N, E, H, D, 2, 2) if proj else b_gat(N, E, H, D, 2, 2, args.alpha_out),
    }
    B_step = sum(B.values())
    value = B_step / (ms_step * 1e-3) / 1e9
    B_unique = dict(B, spmm=b_unique_spmm(N, M, E, F, 2, 2), spmm_t=b_unique_spmm(M, N, E, F, 2, 2),
                    gat_aggregate=b_unique_gat(N, M, E, H, D, 2, 2) - (4 * M * H - 4 * H * D if proj else 0))
    FLOP = {"spmm": 2 * E * F, "spmm_t": 2 * E * F,
            "gat_aggregate": (4 if proj else 2) * E * H * D + 8 * E * H}
    ops = {}
    for op in OPS:
        ms = op_ms[op]
        ok = ms > 0
        ops[op] = dict(ms=ms, ms_median=float(np.median(op_all[op])), ms_min=min(op_all[op]),
                       algorithmic_GB=B[op] / 1e9,
                       eff_GBps=(B[op] / (ms * 1e-3) / 1e9) if ok else None,
                       pct_peak=(B[op] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS) if ok else None,
                       unique_GBps=(B_unique[op] / (ms * 1e-3) / 1e9) if ok else None,
                       GFLOPps=(FLOP[op] / (ms * 1e-3) / 1e9) if ok and op in FLOP else None,
                       edges_per_s=(E / (ms * 1e-3)) if ok and not op.startswith("plan") else None)
    # dominant kernel: the largest device time per step; its algorithmic bytes
    # are its own edges and output rows (per nonzero: index, value, one feature
    # row; per row: row pointer and the output row)
    e_sp, r_sp = 8 + F * 2, 4 + F * 2
    e_gat, r_gat = 4 + (0 if proj else 4 * H) + H * D * 2, 4 + 4 * H + H * D * 2
    kbytes = {
        "spmm": us["E_long"] * e_sp + us["R_long"] * r_sp,
        "spmm_t": us_t["E_long"] * e_sp + us_t["R_long"] * r_sp,
        gat_k: us["E_long"] * e_gat + us["R_long"] * r_gat,
    }
    dom = max(kbytes, key=lambda k: kernels.get(k, {"total_ms": 0})["total_ms"])
    dom_op = {"spmm": "spmm", "spmm_t": "spmm_t", gat_k: "gat_aggregate"}[dom]
    dom_bytes = kbytes[dom]
    dom_launches = [ms for name, ms in roof_trace if name == dom]
    dom_ms = sum(dom_launches) / len(dom_launches)
    eff = dom_bytes / (dom_ms * 1e-3) / 1e9
    # measured HBM bytes: the probe under rocprofv3 in this run, else the committed record
    counters, why = (None, "--no-live-counters") if args.no_live_counters else live_counters(args)
    if counters is None:
        log(f"live counters unavailable ({why}); falling back on the committed record")
        counters = recorded_traffic(cfg["name"])
    tr = kernel_traffic(counters, dom) if counters else None
    hbm_rate = tr["bytes"] / (dom_ms * 1e-3) / 1e9 if tr else None
    roofline = dict(
        bound="hbm", kernel=dom, achieved=hbm_rate, peak=HBM_PEAK_GBPS, unit="GB/s",
        frac=hbm_rate / HBM_PEAK_GBPS if tr else None, traffic=tr["bytes"] if tr else None,
        basis=("achieved = measured HBM bytes of one launch (rocprofv3 FETCH_SIZE + WRITE_SIZE of the "
               "kernel's dispatch in one step of this workload, each scaled by what the counter reads "
               "for a copy of known size) / the kernel's mean launch time over the timed region (HIP "
               "events on its stream)"),
        avg_ms=dom_ms, launches_timed=len(dom_launches),
        effective_GBps=eff, effective_frac=eff / HBM_PEAK_GBPS, algorithmic_bytes_per_launch=dom_bytes,
        effective_note=("algorithmic bytes (one gather of the feature row per nonzero) / time: above "
                        "the HBM peak when hot rows are served from L2, so not an HBM fraction"),
        compulsory_GBps=B_unique[dom_op] / (op_ms[dom_op] * 1e-3) / 1e9,
        traffic_detail=(dict(tr, source=counters.get("source"), fetch_scale=counters["fetch_scale"],
                             write_scale=counters["write_scale"],
                             hbm_over_algorithmic=tr["bytes"] / dom_bytes) if tr else None),
        counters_unavailable=None if counters else why)
    step_hbm = None
    if counters:
        sb = counters["step_bytes"]
        step_hbm = dict(bytes=sb, GBps=sb / (ms_step * 1e-3) / 1e9, frac=sb / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                        note="calibrated FETCH_SIZE + WRITE_SIZE summed over every dispatch of one step / step time",
                        calibration=counters["calibration"],
                        per_launch_GB={f"{i:02d} {d['launch']}": round((d["fetch_bytes"] + d["write_bytes"]) / 1e9, 4)
                                       for i, d in enumerate(counters["step"])})

    # Entry points outside the fused forward step, timed on the same inputs:
    # the standalone SDDMM + edge softmax (alpha written), the fused
    # aggregation with alpha written for the backward pass, and the GSpMM
    # mean and max reduces (max with the int32 edge id of every output).
    alpha_buf = torch.empty((E, H), dtype=torch.float32, device=dev)

    def time_op(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps



    def time_op_kernels(fn, reps=5):
        """Average time of fn and of each library kernel it launches."""
        ms = time_op(fn, reps)
        cg.trace_enable(4096)
        cg.trace_reset()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        per_k = {}
        for name, kms in cg.trace_read():
            per_k[name] = per_k.get(name, 0.0) + kms / reps
        cg.trace_enable(0)
        return ms, per_k

    ms_gat_given, k_gat_given = time_op_kernels(
        lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan, out=Yg))
    # The standalone softmax on the step's plan and on a plain one (a plan is the caller's
    # choice per call): under column slicing 75% of the edges sit in split rows whose scores
    # are parked and rewritten, which a plain plan mostly avoids; `ms` is the faster of the two.
    plan_soft = plan if args.plain_plans else cg.Plan(rowptr, E, max_feat=H, max_heads=H,
                                                      group_size=args.group_size)
    soft_runs = {}
    for tag, p_ in (("step_plan", plan), ("plain_plan", plan_soft)):
        soft_runs[tag] = time_op_kernels(lambda: cg.sddmm_edge_softmax(rowptr, col, s_dst, s_src, 0.2, plan=p_,
                                                                       out=alpha_buf))
    soft_plan = min(soft_runs, key=lambda t: soft_runs[t][0])
    ms_soft, k_soft = soft_runs[soft_plan]
    if plan_soft is not plan:
        plan_soft.close()
    ms_gat_a, k_gat_a = time_op_kernels(lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan,
                                                                 out=Yg, alpha_out=alpha_buf))

    # GAT backward (dY random bf16, the forward's alpha), CSR pass + CSC pass
    dYg = up(synth.f32_to_bf16_bits(synth.normal_f32((N, H * D), 4100 + args.config)).view(np.int16),
             torch.bfloat16).view(N, H, D)
    cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan, out=Yg, alpha_out=alpha_buf)
    bwd_out = {"dX": torch.empty((M, H, D), dtype=torch.bfloat16, device=dev),
               "dalpha": torch.empty((E, H), dtype=torch.float32, device=dev),
               "dscore": torch.empty((E, H), dtype=torch.float32, device=dev),
               "ds_dst": torch.empty((N, H), dtype=torch.float32, device=dev),
               "ds_src": torch.empty((M, H), dtype=torch.float32, device=dev),
               "edge_work": torch.empty((E, H, 2), dtype=torch.float32, device=dev)}
    ms_bwd, k_bwd = time_op_kernels(lambda: cg.gat_backward(
        rowptr, col, colptr, row_t, perm, s_dst, s_src, alpha_buf, Xg, dYg, 0.2, plan=plan,
        plan_t=plan_t, out=bwd_out))
    # the same with only a layer's gradients (ds_dst, ds_src, dX; dscore stays in the records)
    lay_out = {k: bwd_out[k] for k in ("dX", "ds_dst", "ds_src", "edge_work")}
    lay_out.update(dalpha=None, dscore=None)
    ms_bwd_l, k_bwd_l = time_op_kernels(lambda: cg.gat_backward(
        rowptr, col, colptr, row_t, perm, s_dst, s_src, alpha_buf, Xg, dYg, 0.2, plan=plan,
        plan_t=plan_t, out=lay_out))
    # a training step's pair without alpha in memory: the forward keeps each row's softmax
    # state (max, 1 / normalizer), the backward rebuilds the weights from it
    st_buf = torch.empty((N, 2, H), dtype=torch.float32, device=dev)
    ms_gat_st, k_gat_st = time_op_kernels(lambda: cg.gat_aggregate_stats(
        rowptr, col, s_dst, Xg, s_src=s_src, negative_slope=0.2, plan=plan, out=Yg, stats_out=st_buf))
    ms_bwd_st, k_bwd_st = time_op_kernels(lambda: cg.gat_backward(
        rowptr, col, colptr, row_t, perm, s_dst, s_src, None, Xg, dYg, 0.2, plan=plan,
        plan_t=plan_t, out=lay_out, row_stats=st_buf))
    # the same pair with the step's projected source scores: the backward takes s_src from one
    # head-score pass over the features (which a layer needs for s_dst anyway)
    ms_gat_stp, _ = time_op_kernels(lambda: cg.gat_aggregate_stats(
        rowptr, col, s_dst, Xg, a_src=a_src, negative_slope=0.2, plan=plan, out=Yg, stats_out=st_buf))
    ms_hs = time_op(lambda: cg.head_scores(Xg, a_src, None))
    s_src_p, _ = cg.head_scores(Xg, a_src, None)
    ms_bwd_stp, _ = time_op_kernels(lambda: cg.gat_backward(
        rowptr, col, colptr, row_t, perm, s_dst, s_src_p, None, Xg, dYg, 0.2, plan=plan,
        plan_t=plan_t, out=lay_out, row_stats=st_buf))
    del lay_out, st_buf, s_src_p
    dot_out = torch.empty((E, H), dtype=torch.float32, device=dev)
    ms_dot, k_dot = time_op_kernels(lambda: cg.sddmm_dot(rowptr, col, dYg, Xg, plan=plan, out=dot_out))
    b_dot = 4 * (N + 1) + 4 * E + N * H * D * 2 + E * H * D * 2 + 4 * E * H
    del bwd_out, dYg, dot_out
    # rows pass: rowptr, col, dY rows, gathered X rows, s_dst, alpha, s_src, dalpha, dscore,
    # the (alpha, dscore) records, ds_dst; cols pass: colptr, row_t, perm, gathered dY rows,
    # one 8H-byte record per edge, dX, ds_src
    b_bwd_rows = (4 * (N + 1) + 4 * E + N * H * D * 2 + E * H * D * 2 + 4 * N * H + 4 * E * H
                  + 4 * E * H + 4 * E * H + 4 * E * H + 8 * E * H + 4 * N * H)
    b_bwd_cols = (4 * (M + 1) + 4 * E + 4 * E + E * H * D * 2 + 4 * E * H + 4 * E * H
                  + M * H * D * 2 + 4 * M * H)
    b_bwd = b_bwd_rows + b_bwd_cols
    b_bwd_l = b_bwd - 8 * E * H                    # no dalpha, no dscore written
    b_bwd_st = b_bwd_l - 4 * E * H + 8 * N * H       # row states read instead of alpha
    b_gat_st = b_gat(N, E, H, D, 2, 2, False) + 8 * N * H

    # activation compression of the layer output Y (N x F bf16) at 2, 3, 4 bits, groups of F
    codec = {}
    for bits in (2, 3, 4):
        words, nst = cg.act_codec_size(N, F, bits, F)
        cbuf = torch.empty(words, dtype=torch.int64, device=dev)
        sbuf = torch.empty(nst, dtype=torch.float32, device=dev)
        dbuf = torch.empty((N, F), dtype=torch.bfloat16, device=dev)
        ms_c = time_op(lambda: cg.act_compress(Y, bits, F, 1234, codes=cbuf, stats=sbuf))
        ms_d = time_op(lambda: cg.act_decompress(cbuf, sbuf, N, F, bits, F, out=dbuf))
        b_raw, b_cmp = N * F * 2, words * 8 + nst * 4
        codec[f"{bits}bit"] = dict(compress_ms=ms_c, decompress_ms=ms_d,
                                   compress_GBps=(b_raw + b_cmp) / (ms_c * 1e-3) / 1e9,
                                   decompress_GBps=(b_raw + b_cmp) / (ms_d * 1e-3) / 1e9,
                                   ratio_vs_fp32=(N * F * 4) / b_cmp, ratio_vs_bf16=b_raw / b_cmp)
        del cbuf, sbuf, dbuf

    ms_mean = time_op(lambda: cg.gspmm(rowptr, col, val, X, "mean", plan=plan, out=Y))
    arg_buf = torch.empty((N, F), dtype=torch.int32, device=dev)
    ms_max = time_op(lambda: cg.gspmm(rowptr, col, val, X, "max", plan=plan, out=Y,
                                      return_arg=True, arg=arg_buf))
    del arg_buf
    b_mean = b_spmm(N, M, E, F, 2, 2)
    b_max = b_mean + 4 * N * F
    b_soft = 4 * (N + 1) + 4 * E + 4 * N * H + 4 * E * H + 4 * E * H
    b_gat_a = b_gat(N, E, H, D, 2, 2, True)
    extra_ops = {
        "sddmm_edge_softmax": dict(ms=ms_soft, algorithmic_GB=b_soft / 1e9,
                                   eff_GBps=b_soft / (ms_soft * 1e-3) / 1e9,
                                   edges_per_s=E / (ms_soft * 1e-3), kernels_ms=k_soft, plan=soft_plan,
                                   ms_by_plan={t: v[0] for t, v in soft_runs.items()}),
        "gat_aggregate_given_scores": dict(ms=ms_gat_given, algorithmic_GB=b_gat(N, E, H, D, 2, 2, False) / 1e9,
                                           eff_GBps=b_gat(N, E, H, D, 2, 2, False) / (ms_gat_given * 1e-3) / 1e9,
                                           edges_per_s=E / (ms_gat_given * 1e-3), kernels_ms=k_gat_given),
        "gat_aggregate_with_alpha": dict(ms=ms_gat_a, algorithmic_GB=b_gat_a / 1e9,
                                         eff_GBps=b_gat_a / (ms_gat_a * 1e-3) / 1e9,
                                         edges_per_s=E / (ms_gat_a * 1e-3), kernels_ms=k_gat_a,
                                         over_given_scores_ms=ms_gat_a - ms_gat_given),
        "gat_backward": dict(ms=ms_bwd, algorithmic_GB=b_bwd / 1e9,
                             eff_GBps=b_bwd / (ms_bwd * 1e-3) / 1e9,
                             edges_per_s=E / (ms_bwd * 1e-3),
                             kernels_ms=k_bwd,
                             rows_pass_GBps=b_bwd_rows / (k_bwd.get("gat_bwd_rows", 0) * 1e-3) / 1e9
                             if k_bwd.get("gat_bwd_rows") else None,
                             cols_pass_GBps=b_bwd_cols / ((k_bwd.get("gat_bwd_cols", 0)
                                                           + k_bwd.get("gat_bwd_cols_tiny", 0)) * 1e-3) / 1e9
                             if k_bwd.get("gat_bwd_cols") else None),
        "gat_backward_layer_gradients": dict(
            ms=ms_bwd_l, algorithmic_GB=b_bwd_l / 1e9, eff_GBps=b_bwd_l / (ms_bwd_l * 1e-3) / 1e9,
            edges_per_s=E / (ms_bwd_l * 1e-3), kernels_ms=k_bwd_l,
            note="dalpha and dscore not written: ds_dst, ds_src, dX and the (alpha, dscore) records"),
        "gat_training_pair_row_states": dict(
            forward_ms=ms_gat_st, backward_ms=ms_bwd_st, ms=ms_gat_st + ms_bwd_st,
            forward_algorithmic_GB=b_gat_st / 1e9, backward_algorithmic_GB=b_bwd_st / 1e9,
            forward_kernels_ms=k_gat_st, backward_kernels_ms=k_bwd_st,
            with_alpha_ms=ms_gat_a + ms_bwd_l,
            projected_scores=dict(forward_ms=ms_gat_stp, head_scores_ms=ms_hs, backward_ms=ms_bwd_stp,
                                  ms=ms_gat_stp + ms_hs + ms_bwd_stp),
            note="forward with each row's softmax state instead of alpha, backward rebuilding the "
                 "weights (layer gradients only); with_alpha_ms: the same pair through alpha; "
                 "projected_scores: the forward forms s_src from the gathered rows, the backward "
                 "takes it from a head-score pass"),
        "act_codec": codec,
        "sddmm_dot": dict(ms=ms_dot, algorithmic_GB=b_dot / 1e9,
                          eff_GBps=b_dot / (ms_dot * 1e-3) / 1e9, edges_per_s=E / (ms_dot * 1e-3)),
        "gspmm_mean": dict(ms=ms_mean, algorithmic_GB=b_mean / 1e9,
                           eff_GBps=b_mean / (ms_mean * 1e-3) / 1e9,
                           edges_per_s=E / (ms_mean * 1e-3)),
        "gspmm_max_with_arg": dict(ms=ms_max, algorithmic_GB=b_max / 1e9,
                                   eff_GBps=b_max / (ms_max * 1e-3) / 1e9,
                                   edges_per_s=E / (ms_max * 1e-3)),
    }
    # Warm mode: the same call back to back, so what the previous call left in
    # L2 and the memory-side cache is reused (inside the step every operator
    # follows gigabytes of unrelated traffic, which is the cold case).
    def warm(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        evs[0].record()
        for i in range(reps):
            fn()
            evs[i + 1].record()
        torch.cuda.synchronize()
        t = [evs[i].elapsed_time(evs[i + 1]) for i in range(reps)]
        return dict(ms_median=float(np.median(t)), ms_min=min(t))
    warm_ops = {
        "spmm": warm(lambda: cg.spmm(rowptr, col, val, X, plan=plan, out=Y)),
        "spmm_t": warm(lambda: cg.spmm_t(colptr, row_t, val_t, Gt, plan_t=plan_t, out=dX)),
        "gat_aggregate": warm(lambda: cg.gat_aggregate_proj(rowptr, col, s_dst, a_src, Xg, 0.2, plan=plan,
                                                            out=Yg)) if proj else
        warm(lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan,
                                                       out=Yg)),
    }
    for op, w in warm_ops.items():
        w["eff_GBps"] = B[op] / (w["ms_median"] * 1e-3) / 1e9
    # achievable-bandwidth ceiling: a plain 1 GiB device-to-device copy
    cp_src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    cp_dst = torch.empty_like(cp_src)
    cp = warm(lambda: cp_dst.copy_(cp_src), reps=5)
    copy_GBps = 2 * (1 << 30) / (cp["ms_median"] * 1e-3) / 1e9
    del cp_src, cp_dst
    log(f"warm (back to back): " + ", ".join(f"{k} {v['ms_median']:.3f} ms" for k, v in warm_ops.items())
        + f"; 1 GiB copy {copy_GBps:.0f} GB/s")

    codec_txt = ", ".join("%s %.3f/%.3f" % (k, v["compress_ms"], v["decompress_ms"]) for k, v in codec.items())
    log(f"extra: sddmm_edge_softmax {ms_soft:.3f} ms, gat_aggregate+alpha {ms_gat_a:.3f} ms, "
        f"gspmm mean {ms_mean:.3f} ms, max+arg {ms_max:.3f} ms, sddmm_dot {ms_dot:.3f} ms, "
        f"codec (compress/decompress) {codec_txt} ms, "
        f"gat backward {ms_bwd:.3f} ms "
        f"({', '.join(f'{k} {v:.3f}' for k, v in k_bwd.items())}), "
        f"layer gradients only {ms_bwd_l:.3f} ms "
        f"({', '.join(f'{k} {v:.3f}' for k, v in k_bwd_l.items())}); "
        f"training pair through row states {ms_gat_st:.3f} + {ms_bwd_st:.3f} ms "
        f"(through alpha {ms_gat_a:.3f} + {ms_bwd_l:.3f} ms; projected scores {ms_gat_stp:.3f} + "
        f"{ms_hs:.3f} + {ms_bwd_stp:.3f} ms)")

    inference = None if args.no_inference else run_inference(cg, synth, dev, time_op_kernels,
                                                             sliced=not args.plain_plans)

    out = {
        "metric": METRIC, "value": value, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded R-MAT graph, normal features; no dataset)",
        "config": {"workload": (f"{cfg['name']}: R-MAT a=0.57 b=0.19 c=0.19, N={N}, nnz={E} "
                                f"incl. self-loops, 4 hub rows (100k-300k), GCN F={F} bf16, "
                                f"GAT H={H} x D={D} bf16, fp32 accumulation"),
                   "n_nodes": N, "nnz": E, "F": F, "H": H, "D": D, "feature_dtype": "bf16",
                   "accumulate": "f32", "group_size": info["group_size"],
                   "balancer": info["mode_name"],
                   "column_slices": None if args.plain_plans else
                   f"8 column ranges, rows over {SLICE_MIN} nonzeros sliced, one unit list per XCD",
                   "alpha_out": bool(args.alpha_out),
                   "gat_source_scores": ("projected from the gathered feature rows in the kernel: "
                                         "s_src[j] = X[j] a_src, a_src N(0, 1/D) (cogdl_gat_aggregate_proj)"
                                         if proj else "given N x H fp32 ~N(0,1) (cogdl_gat_aggregate)")},
        "pct_peak": value / HBM_PEAK_GBPS,
        "edges_per_s": 3 * E / (ms_step * 1e-3),
        "edges_per_s_note": "nonzeros aggregated per second over the three gathers (SpMM, SpMM^T, GAT)",
        "ops": ops,
        "ops_timing": ("ops and kernels: mean, median and min over an instrumented pass of the same "
                       "number of steps run after the timed region (events between operators and "
                       "around every launch; its step time is ms_per_step_instrumented); each "
                       "operator is cold there (it follows gigabytes of other traffic in the step). "
                       "ops_warm: the same call repeated back to back. roofline.avg_ms: the timed "
                       "region's own launches of that kernel, timed by events placed around the "
                       "SpMM, SpMM^T and GAT launches only"),
        "ms_per_step_instrumented": ms_step_instr,
        "ops_warm": warm_ops,
        "copy_GBps": copy_GBps,
        "ops_outside_step": extra_ops,
        "kernels": kernels,
        "roofline": roofline,
        "step_hbm": step_hbm,
        "inference": inference,
    }
    if not args.no_cpu_baseline:
        log("CPU baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(g, X_bits, Xg_bits, sd, ss, H, D, F, args.cpu_seconds,
                                           a_src=a_src_h if proj else None)
        log(f"CPU baseline {out['cpu_baseline']['value']:.2f} GB/s on {out['cpu_baseline']['cores']} threads")
    plan.close()
    plan_t.close()
    if not args.no_workloads:
        # The other workloads' own operators (workloads 1-4 in their own dtypes and plans),
        # each with its time, rates, HBM bytes from counters and the CPU oracle's rate.
        wl_hbm, why = (None, "--no-live-counters") if args.no_live_counters else live_workload_counters(args)
        if wl_hbm is None:
            log(f"live workload counters unavailable ({why}); falling back on the committed record")
        out["workloads"] = run_workloads(reps=args.wl_reps, warm_reps=2, cpu=not args.no_cpu_baseline,
                                         cpu_budget_s=1.0, hbm=wl_hbm, emit=lambda r: None)
        out["workloads_note"] = ("workloads 1-4 (cold: a 1 GiB buffer written before each call; warm: back to "
                                 "back), median and minimum of wl_reps calls; hbm_* from the counters of one cold "
                                 "call (hbm_source); cpu_oracle: the fp64 oracle on all host threads (and one thread "
                                 "for workloads 1-2); cache_resident: the gathered table fits the 256 MB Infinity "
                                 "Cache, so algorithmic rates can exceed the HBM peak there")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
