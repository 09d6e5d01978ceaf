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
    ap.add_argument("--alpha-out", action="store_true", help="also write alpha in the GAT step")
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

# The step's candidate roofline kernels: the sources that define each one, its
# instantiation on the benchmark workload (bf16 in and out, 16-byte vectors,
# one chunk, buffer gathers), and which of that kernel's dispatches in one step
# is the op (the SpMM and the transposed SpMM share an instantiation).
ROOFLINE_KERNELS = {
    "spmm": dict(files=["common.hpp", "internal.hpp", "spmm_kernel.hpp", "spmm.hip"],
                 name="void k_spmm<bf16_t, bf16_t, 8, 1, true, false, false>", per_step=2, index=0),
    "spmm_t": dict(files=["common.hpp", "internal.hpp", "spmm_kernel.hpp", "spmm.hip"],
                   name="void k_spmm<bf16_t, bf16_t, 8, 1, true, false, false>", per_step=2, index=1),
    "gat": dict(files=["common.hpp", "internal.hpp", "gat_kernel.hpp", "gat.hip"],
                name="void k_gat<bf16_t, bf16_t, 8, 1, true, false>", per_step=1, index=0),
}


def kernel_source_sha(kernel: str) -> str:
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    csrc = os.path.join(here, "paper_2103_00959_amd", "csrc")
    files = ROOFLINE_KERNELS[kernel]["files"]
    return hashlib.sha256(b"".join(open(os.path.join(csrc, f), "rb").read() for f in files)).hexdigest()[:16]


def recorded_traffic(workload: str, kernel: str, profiles_dir: str | None = None):
    """HBM bytes of one launch of the step's kernel `kernel` from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary (scaled by the copy calibration;
    the dispatch of the timed step of a --warmup 1 run), or None when that
    kernel's sources changed since the counters were taken."""
    if profiles_dir is None:
        profiles_dir = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles")
    path = os.path.join(profiles_dir, f"{workload}_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    shas = rec.get("source_sha16")
    if not isinstance(shas, dict) or shas.get(kernel) != kernel_source_sha(kernel):
        return None
    spec = ROOFLINE_KERNELS[kernel]
    disp = rec["kernels"].get(spec["name"])
    if not disp:
        return None
    i = spec["per_step"] * rec.get("warmup", 1) + spec["index"]
    if i >= len(disp):
        return None
    d = disp[i]
    return dict(bytes=d["fetch_bytes"] + d["write_bytes"], fetch_bytes=d["fetch_bytes"],
                write_bytes=d["write_bytes"], l2_hit=d.get("l2_hit"), kernel=spec["name"], dispatch=i,
                dur_ms=d["dur_ms"], source=os.path.basename(path))


def cpu_baseline(g, X_bits, Xg_bits, sd, ss, H, D, F, budget_s):
    """Time the oracle (fp64, all host threads) on a random row sample of the
    SpMM and GAT steps, growing the sample until the budget is spent."""
    import oracle
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    oracle.set_threads(threads)
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
        bytes_total += b_spmm(sel.size, g.n_cols, e, F, 2, 2) + b_gat(sel.size, e, H, D, 2, 2, False)
        edges_total += 2 * e
        chunk = min(chunk * 2, 200000)
    return dict(value=bytes_total / t_total / 1e9, unit="GB/s", cores=threads, kind="oracle",
                cpu=cpu_model(),
                sample=(f"SpMM (F=256 bf16) + fused GAT (4x64 bf16) on {done_rows} random rows "
                        f"({edges_total // 2} nonzeros each) of the same graph, fp64 oracle"),
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


def run_workloads(reps=20, warm_reps=3, cpu=True, cpu_budget_s=2.0):
    """Each workload's operators in its own configuration (fp32 features; column-sliced plans
    on AUTO with the default group size), one JSON line per (workload, op).  Cold: a 1 GiB buffer is
    written before every timed call, so L2 and the Infinity Cache hold none of its inputs;
    warm: the same call back to back.  Median and minimum of `reps` calls after `warm_reps`
    untimed ones; plan creation and the transpose are preprocessing, reported on their own.
    Each line also carries the compulsory-byte rate, GFLOP/s, whether the gathered table fits
    the 256 MB Infinity Cache, a 1 GiB copy's rate (the achievable ceiling), the HBM bytes
    of one cold call from the committed rocprofv3 counters of this mode (when the library
    sources are unchanged since), and the fp64 CPU oracle's rate on the same op (all host
    threads; also one thread for workloads 1 and 2, whose ops the oracle does whole)."""
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
    hbm = recorded_workload_traffic()
    threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    cpu_name = cpu_model()
    if cpu:
        import oracle

    def times(fn):
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
               "hbm_GBps": None, "l2_hit": None, "cpu_oracle": cpu_rec}
        h = hbm.get(f"{cfg['name']}/{op}") if hbm else None
        if h:
            out["hbm_GB"] = (h["fetch_bytes"] + h["write_bytes"]) / 1e9
            out["hbm_GBps"] = (h["fetch_bytes"] + h["write_bytes"]) / (mc * 1e-3) / 1e9
            out["l2_hit"] = h.get("l2_hit")
        print(json.dumps(out), flush=True)
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


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path has no "
              f"multi-GPU mode in this build", file=sys.stderr)
        sys.exit(2)
    if args.workloads:
        run_workloads(reps=args.reps, warm_reps=args.warm_reps, cpu=not args.no_cpu_baseline)
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
    X32 = synth.normal_f32((M, F), 2000 + args.config)
    X_bits = synth.f32_to_bf16_bits(X32)
    del X32
    G_bits = synth.f32_to_bf16_bits(synth.normal_f32((N, F), 4000 + args.config))
    Xg_bits = synth.f32_to_bf16_bits(synth.normal_f32((M, H * D), 2100 + args.config))
    rng = np.random.default_rng(3000 + args.config)
    sd = rng.standard_normal((N, H), dtype=np.float32)
    ss = rng.standard_normal((M, H), dtype=np.float32)
    log(f"features ready in {time.time() - t0:.1f}s")

    dev = torch.device("cuda:0")

    def up(a, dt=None):
        t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return t.view(dt) if dt is not None else t

    rowptr, col, val = up(g.rowptr), up(g.col), up(g.val)
    X = up(X_bits.view(np.int16), torch.bfloat16)
    Gt = up(G_bits.view(np.int16), torch.bfloat16)
    Xg = up(Xg_bits.view(np.int16), torch.bfloat16).view(M, H, D)
    s_dst, s_src = up(sd), up(ss)
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
        cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan, out=Yg,  # a5-a7
                         alpha_out=alpha)
        mark(6)

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
    ROOF = ("spmm", "spmm_t", "gat")
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
        "gat_aggregate": b_gat(N, E, H, D, 2, 2, args.alpha_out),
    }
    B_step = sum(B.values())
    value = B_step / (ms_step * 1e-3) / 1e9
    B_unique = dict(B, spmm=b_unique_spmm(N, M, E, F, 2, 2), spmm_t=b_unique_spmm(M, N, E, F, 2, 2),
                    gat_aggregate=b_unique_gat(N, M, E, H, D, 2, 2))
    FLOP = {"spmm": 2 * E * F, "spmm_t": 2 * E * F, "gat_aggregate": 2 * E * H * D + 8 * E * H}
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
    e_gat, r_gat = 4 + 4 * H + H * D * 2, 4 + 4 * H + H * D * 2
    kbytes = {
        "spmm": us["E_long"] * e_sp + us["R_long"] * r_sp,
        "spmm_t": us_t["E_long"] * e_sp + us_t["R_long"] * r_sp,
        "gat": us["E_long"] * e_gat + us["R_long"] * r_gat,
    }
    dom = max(kbytes, key=lambda k: kernels.get(k, {"total_ms": 0})["total_ms"])
    dom_bytes = kbytes[dom]
    dom_launches = [ms for name, ms in roof_trace if name == dom]
    dom_ms = sum(dom_launches) / len(dom_launches)
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    tr = recorded_traffic(cfg["name"], dom)
    roofline = dict(bound="hbm", kernel=dom, achieved=achieved, peak=HBM_PEAK_GBPS, unit="GB/s",
                    frac=achieved / HBM_PEAK_GBPS, traffic=(tr["bytes"] if tr else None),
                    algorithmic_bytes_per_launch=dom_bytes, avg_ms=dom_ms,
                    traffic_detail=tr)

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

    ms_soft = time_op(lambda: cg.sddmm_edge_softmax(rowptr, col, s_dst, s_src, 0.2, plan=plan,
                                                    out=alpha_buf))
    ms_gat_a = time_op(lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan,
                                                out=Yg, alpha_out=alpha_buf))
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

    # GAT backward (dY random bf16, the forward's alpha), CSR pass + CSC pass
    dYg = up(synth.f32_to_bf16_bits(synth.normal_f32((N, H * D), 4100 + args.config)).view(np.int16),
             torch.bfloat16).view(N, H, D)
    cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan, out=Yg, alpha_out=alpha_buf)
    bwd_out = {"dX": torch.empty((M, H, D), dtype=torch.bfloat16, device=dev),
               "dalpha": torch.empty((E, H), dtype=torch.float32, device=dev),
               "dscore": torch.empty((E, H), dtype=torch.float32, device=dev),
               "ds_dst": torch.empty((N, H), dtype=torch.float32, device=dev),
               "ds_src": torch.empty((M, H), dtype=torch.float32, device=dev)}
    ms_bwd, k_bwd = time_op_kernels(lambda: cg.gat_backward(
        rowptr, col, colptr, row_t, perm, s_dst, s_src, alpha_buf, Xg, dYg, 0.2, plan=plan,
        plan_t=plan_t, out=bwd_out))
    dot_out = torch.empty((E, H), dtype=torch.float32, device=dev)
    ms_dot, k_dot = time_op_kernels(lambda: cg.sddmm_dot(rowptr, col, dYg, Xg, plan=plan, out=dot_out))
    b_dot = 4 * (N + 1) + 4 * E + N * H * D * 2 + E * H * D * 2 + 4 * E * H
    del bwd_out, dYg, dot_out
    b_bwd_rows = (4 * (N + 1) + 4 * E + N * H * D * 2 + E * H * D * 2 + 4 * N * H + 4 * E * H
                  + 4 * E * H + 4 * E * H + 4 * E * H + 4 * N * H)
    b_bwd_cols = (4 * (M + 1) + 4 * E + 4 * E + E * H * D * 2 + 4 * E * H + 4 * E * H
                  + M * H * D * 2 + 4 * M * H)
    b_bwd = b_bwd_rows + b_bwd_cols

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
                                   edges_per_s=E / (ms_soft * 1e-3)),
        "gat_aggregate_with_alpha": dict(ms=ms_gat_a, algorithmic_GB=b_gat_a / 1e9,
                                         eff_GBps=b_gat_a / (ms_gat_a * 1e-3) / 1e9,
                                         edges_per_s=E / (ms_gat_a * 1e-3)),
        "gat_backward": dict(ms=ms_bwd, algorithmic_GB=b_bwd / 1e9,
                             eff_GBps=b_bwd / (ms_bwd * 1e-3) / 1e9,
                             edges_per_s=E / (ms_bwd * 1e-3),
                             kernels_ms=k_bwd,
                             rows_pass_GBps=b_bwd_rows / (k_bwd.get("gat_bwd_rows", 0) * 1e-3) / 1e9
                             if k_bwd.get("gat_bwd_rows") else None,
                             cols_pass_GBps=b_bwd_cols / ((k_bwd.get("gat_bwd_cols", 0)
                                                           + k_bwd.get("gat_bwd_cols_tiny", 0)) * 1e-3) / 1e9
                             if k_bwd.get("gat_bwd_cols") else None),
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
        "gat_aggregate": warm(lambda: cg.gat_aggregate(rowptr, col, s_dst, s_src, Xg, 0.2, plan=plan,
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
        f"({', '.join(f'{k} {v:.3f}' for k, v in k_bwd.items())})")

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
                   "alpha_out": bool(args.alpha_out)},
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
        "inference": inference,
    }
    if not args.no_cpu_baseline:
        log("CPU baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(g, X_bits, Xg_bits, sd, ss, H, D, F, args.cpu_seconds)
        log(f"CPU baseline {out['cpu_baseline']['value']:.2f} GB/s on {out['cpu_baseline']['cores']} threads")
    plan.close()
    plan_t.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
