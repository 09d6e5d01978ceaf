"""Seeded synthetic graphs and features shaped like the CogDL paper's workloads.

The paper measures its sparse operators on Reddit, Yelp, Flickr and ogbn-style
graphs (section 3.2, Figure 1; section 3.3, Table 4; dataset statistics in the
node-classification dataset table).  None of those datasets is used here:
every input is drawn from a seeded random-graph model with the node count,
edge count and degree skew of the corresponding workload.

This module holds input generation only (graph models, the graph normalization
that produces the edge values, and feature sampling).  It contains none of the
operators themselves; both the HIP library's tests/benchmark and the CPU
oracle's tests take their inputs from here.

Recipes (numpy PCG64 generators, one seed per stream):
  * Erdos-Renyi G(n, m): m distinct unordered pairs, no self pairs, stored in
    both directions.
  * R-MAT (Graph500 style, a=0.57, b=0.19, c=0.19, d=0.05): each of the
    ``scale`` levels picks a quadrant from a 16-bit uniform draw; endpoints
    >= n are rejected, self pairs dropped, duplicates removed, and sampling
    continues until exactly the target number of distinct directed edges
    exists (a seeded random surplus is dropped).  A seeded random permutation
    of vertex ids then removes the id locality of the model.
  * Chung-Lu with a bounded power law: per-node weights from a Pareto law on
    [1, dmax] whose exponent is solved so that the mean is the target mean
    degree; row degrees are the weights scaled to the exact edge total; columns
    are drawn proportionally to the same weights, distinct within a row and
    never equal to the row.
  * Planted hubs: chosen node ids whose rows hold exactly the given number of
    distinct uniform columns (R-MAT samples on those rows are rejected).
  * Self-loops (one per node) are added where a workload says so; columns are
    sorted inside each row.
  * Edge values: symmetric normalization R^-1/2 (A+I) C^-1/2 (R, C = row and
    column counts of the pattern, equal to D^-1/2 (A+I) D^-1/2 on undirected
    graphs) or row normalization 1/d_i, computed in float64, stored as float32.
  * Features: standard normal float32; bf16 copies are the round-to-nearest-
    even of those float32 values.
"""
from __future__ import annotations

import dataclasses
import os
import sys
import time

import numpy as np

RMAT_ABC = (0.57, 0.19, 0.19)


@dataclasses.dataclass
class Graph:
    """CSR graph: row i aggregates from columns col[rowptr[i]:rowptr[i+1]]."""
    rowptr: np.ndarray       # int32 [n_rows + 1]
    col: np.ndarray          # int32 [nnz]
    val: np.ndarray | None   # float32 [nnz]
    n_rows: int
    n_cols: int

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr.astype(np.int64))


# ----------------------------------------------------------------- helpers

def _csr_from_keys(keys: np.ndarray, n_rows: int, n_cols: int) -> Graph:
    """Sorted unique int64 keys row*n_cols+col -> CSR with sorted columns."""
    rows = keys // n_cols
    col = (keys - rows * n_cols).astype(np.int32)
    counts = np.bincount(rows, minlength=n_rows)
    rowptr = np.zeros(n_rows + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return Graph(rowptr.astype(np.int32), col, None, n_rows, n_cols)


def _self_loop_keys(n: int) -> np.ndarray:
    i = np.arange(n, dtype=np.int64)
    return i * n + i


def _drop_surplus(keys: np.ndarray, target: int, rng: np.random.Generator) -> np.ndarray:
    if keys.size > target:
        drop = rng.choice(keys.size, size=keys.size - target, replace=False)
        keys = np.delete(keys, drop)
    return keys


# -------------------------------------------------------------- Erdos-Renyi

def erdos_renyi(n: int, m_pairs: int, seed: int, self_loops: bool = True) -> Graph:
    """Undirected G(n, m) stored in both directions, plus self-loops."""
    rng = np.random.default_rng(seed)
    pairs = np.empty(0, dtype=np.int64)
    while pairs.size < m_pairs:
        need = (m_pairs - pairs.size) * 2 + 16
        u = rng.integers(0, n, size=need, dtype=np.int64)
        v = rng.integers(0, n, size=need, dtype=np.int64)
        keep = u != v
        lo, hi = np.minimum(u, v)[keep], np.maximum(u, v)[keep]
        pairs = np.unique(np.concatenate([pairs, lo * n + hi]))
    pairs = _drop_surplus(pairs, m_pairs, rng)
    lo, hi = pairs // n, pairs % n
    keys = [lo * n + hi, hi * n + lo]
    if self_loops:
        keys.append(_self_loop_keys(n))
    return _csr_from_keys(np.unique(np.concatenate(keys)), n, n)


# -------------------------------------------------------------------- R-MAT

def _quadrant_table(a: float, b: float, c: float) -> np.ndarray:
    """16-bit uniform draw -> quadrant code (src_bit << 1) | dst_bit."""
    r = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
    q = np.full(65536, 3, dtype=np.uint8)
    q[r < a + b + c] = 2
    q[r < a + b] = 1
    q[r < a] = 0
    return q


def _rmat_sample(rng, count: int, scale: int, table: np.ndarray):
    src = np.zeros(count, dtype=np.int64)
    dst = np.zeros(count, dtype=np.int64)
    draws = np.frombuffer(rng.bytes(2 * count * scale), dtype=np.uint16).reshape(scale, count)
    for lvl in range(scale):
        q = table[draws[lvl]]
        src <<= 1
        dst <<= 1
        src |= q >> 1
        dst |= q & 1
    return src, dst


def rmat_keys(n: int, scale: int, target: int, rng: np.random.Generator, perm: np.ndarray,
              exclude_rows: np.ndarray | None = None, abc=RMAT_ABC,
              chunk: int = 1 << 23) -> np.ndarray:
    """Exactly ``target`` distinct directed (src, dst) keys src*n+dst, ids permuted
    by ``perm``, no self pairs, rows in ``exclude_rows`` rejected."""
    table = _quadrant_table(*abc)
    excluded = None
    if exclude_rows is not None and len(exclude_rows):
        excluded = np.zeros(n, dtype=bool)
        excluded[exclude_rows] = True
    keys = np.empty(0, dtype=np.int64)
    want = target
    while keys.size < target:
        parts = []
        drawn = 0
        while drawn < want:
            cnt = min(chunk, want - drawn)
            s, d = _rmat_sample(rng, cnt, scale, table)
            ok = (s < n) & (d < n)
            s, d = perm[s[ok]], perm[d[ok]]
            ok = s != d
            if excluded is not None:
                ok &= ~excluded[s]
            parts.append(s[ok] * n + d[ok])
            drawn += cnt
        new = np.concatenate(parts + [keys])
        keys = np.unique(new)
        # Distinct-edge yield of this round sets the size of the next one.
        got = keys.size
        if got < target:
            frac = max(got / max(new.size, 1), 0.05)
            want = int((target - got) / frac * 1.1) + 1024
    return _drop_surplus(keys, target, rng)


def rmat(n: int, scale: int, unique_edges: int, seed_graph: int, seed_perm: int,
         self_loops: bool = True, hubs: dict | None = None) -> Graph:
    rng = np.random.default_rng(seed_graph)
    perm = np.random.default_rng(seed_perm).permutation(n).astype(np.int64)
    hub_rows = None
    hub_keys = []
    if hubs:
        hub_rows = np.array(sorted(hubs["rows"]), dtype=np.int64)
    rmat_target = unique_edges - (sum(hubs["degrees"]) if hubs else 0)
    keys = rmat_keys(n, scale, rmat_target, rng, perm, exclude_rows=hub_rows)
    if hubs:
        for r, deg in zip(hubs["rows"], hubs["degrees"]):
            cols = rng.choice(n - 1, size=deg, replace=False).astype(np.int64)
            cols[cols >= r] += 1          # skip the self pair
            hub_keys.append(np.int64(r) * n + cols)
    allk = [keys] + hub_keys
    if self_loops:
        allk.append(_self_loop_keys(n))
    return _csr_from_keys(np.unique(np.concatenate(allk)), n, n)


# --------------------------------------------------------------- Chung-Lu

def _bounded_pareto_mean(g: float, lo: float, hi: float) -> float:
    def integral(p):  # int_lo^hi x^p dx
        if abs(p + 1.0) < 1e-12:
            return np.log(hi / lo)
        return (hi ** (p + 1) - lo ** (p + 1)) / (p + 1)
    return integral(1.0 - g) / integral(-g)


def power_law_exponent(mean: float, lo: float, hi: float) -> float:
    """Exponent g of the density x^-g on [lo, hi] with the given mean (bisection)."""
    a, b = 0.01, 4.0          # mean decreases in g
    for _ in range(200):
        m = 0.5 * (a + b)
        if _bounded_pareto_mean(m, lo, hi) > mean:
            a = m
        else:
            b = m
    return 0.5 * (a + b)


def _weighted_draw(rng, cdf: np.ndarray, size: int, table: np.ndarray) -> np.ndarray:
    """Indices i with probability proportional to the weights behind ``cdf``
    (inverse CDF; ``table`` maps 2^k equal buckets of [0, 1) to their first
    candidate index, so a short linear probe finishes the search)."""
    u = rng.random(size)
    idx = table[(u * table.size).astype(np.int64)]
    todo = np.flatnonzero(cdf[idx] <= u)
    while todo.size:
        idx[todo] += 1
        todo = todo[cdf[idx[todo]] <= u[todo]]
    return idx


def chung_lu(n: int, nnz: int, dmin: int, dmax: int, seed: int) -> Graph:
    rng = np.random.default_rng(seed)
    mean = nnz / n
    g = power_law_exponent(mean, dmin, dmax)
    u = rng.random(n)
    one_m = 1.0 - g
    w = (dmin ** one_m + u * (dmax ** one_m - dmin ** one_m)) ** (1.0 / one_m)
    deg = np.clip(np.rint(w * (nnz / w.sum())), dmin, dmax).astype(np.int64)
    diff = nnz - int(deg.sum())
    while diff != 0:
        step = 1 if diff > 0 else -1
        ok = np.flatnonzero((deg + step >= dmin) & (deg + step <= dmax))
        pick = rng.choice(ok, size=min(abs(diff), ok.size), replace=False)
        deg[pick] += step
        diff = nnz - int(deg.sum())
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    cdf[-1] = 1.0 + 1e-12                       # every u < 1 stops at the last index
    table = np.searchsorted(cdf, np.arange(1 << 20) / float(1 << 20), side="right")
    # first round: deg[i] draws for every row; later rounds draw each row's
    # shortfall and merge only the new distinct keys into the sorted key set
    need_rows = np.repeat(np.arange(n, dtype=np.int64), deg)
    keys = np.empty(0, dtype=np.int64)
    while need_rows.size:
        cols = _weighted_draw(rng, cdf, need_rows.size, table)
        ok = cols != need_rows
        new = np.unique(need_rows[ok] * n + cols[ok])
        if keys.size:
            pos = np.searchsorted(keys, new)
            fresh = (pos >= keys.size) | (keys[np.minimum(pos, keys.size - 1)] != new)
            keys = np.insert(keys, pos[fresh], new[fresh])
        else:
            keys = new
        short = deg - np.bincount(keys // n, minlength=n)
        need_rows = np.repeat(np.arange(n, dtype=np.int64), np.maximum(short, 0))
    return _csr_from_keys(keys, n, n)


# --------------------------------------------------------------- weights

def sym_norm_values(g: Graph) -> np.ndarray:
    """R^-1/2 (A+I) C^-1/2 on the stored pattern (which already holds I)."""
    r = g.degrees().astype(np.float64)
    c = np.bincount(g.col, minlength=g.n_cols).astype(np.float64)
    rows = np.repeat(np.arange(g.n_rows), g.degrees())
    return (1.0 / np.sqrt(r[rows] * c[g.col])).astype(np.float32)


def row_norm_values(g: Graph) -> np.ndarray:
    d = g.degrees().astype(np.float64)
    return np.repeat(1.0 / np.maximum(d, 1.0), g.degrees()).astype(np.float32)


# --------------------------------------------------------------- features

def normal_f32(shape, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal(size=shape, dtype=np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


# ------------------------------------------------------------- workloads

CONFIGS = {
    1: dict(name="tiny_gcn_er_2708", kind="er", n=2708, pairs=5278, F=64, weights="sym"),
    2: dict(name="medium_rmat_169343", kind="rmat", n=169343, scale=18, unique=2332486,
            F=128, weights="sym"),
    3: dict(name="dense_chunglu_232965", kind="chunglu", n=232965, nnz=114615892, dmin=1,
            dmax=20000, F=256, weights="row"),
    4: dict(name="gat_rmat_2449029", kind="rmat", n=2449029, scale=22, unique=61859140,
            H=8, D=16, weights=None),
    5: dict(name="skewed_rmat_2400000_hubs", kind="rmat", n=2400000, scale=22,
            unique=120000000, hubs=(100000, 150000, 200000, 300000), F=256, H=4, D=64,
            weights="sym"),
}


def _cache_dir() -> str:
    return os.environ.get("COGDL_SYNTH_CACHE", "/tmp/cogdl_synth_cache")


def _build_graph(k: int) -> Graph:
    cfg = CONFIGS[k]
    if cfg["kind"] == "er":
        g = erdos_renyi(cfg["n"], cfg["pairs"], seed=1000 + k)
    elif cfg["kind"] == "chunglu":
        g = chung_lu(cfg["n"], cfg["nnz"], cfg["dmin"], cfg["dmax"], seed=1000 + k)
    else:
        hubs = None
        if "hubs" in cfg:
            hr = np.random.default_rng(6000 + k).choice(cfg["n"], size=len(cfg["hubs"]),
                                                       replace=False)
            hubs = dict(rows=[int(r) for r in hr], degrees=list(cfg["hubs"]))
        g = rmat(cfg["n"], cfg["scale"], cfg["unique"], seed_graph=1000 + k,
                 seed_perm=5000 + k, hubs=hubs)
    if cfg["weights"] == "sym":
        g.val = sym_norm_values(g)
    elif cfg["weights"] == "row":
        g.val = row_norm_values(g)
    return g


def config_graph(k: int, cache: bool = True, verbose: bool = False) -> Graph:
    """The seeded graph of workload k (1..5), cached as .npy under COGDL_SYNTH_CACHE."""
    cfg = CONFIGS[k]
    d = os.path.join(_cache_dir(), cfg["name"])
    names = ("rowptr", "col", "val")
    if cache and all(os.path.exists(os.path.join(d, f + ".npy")) for f in names[:2]):
        arrs = {f: np.load(os.path.join(d, f + ".npy")) if os.path.exists(
            os.path.join(d, f + ".npy")) else None for f in names}
        return Graph(arrs["rowptr"], arrs["col"], arrs["val"], cfg["n"], cfg["n"])
    t0 = time.time()
    g = _build_graph(k)
    if verbose:
        print(f"[synth] built {cfg['name']}: n={g.n_rows} nnz={g.nnz} in {time.time() - t0:.1f}s",
              flush=True, file=sys.stderr)
    if cache:
        os.makedirs(d, exist_ok=True)
        for f in names:
            a = getattr(g, f)
            if a is not None:
                tmp = os.path.join(d, f"{f}.tmp{os.getpid()}.npy")
                np.save(tmp, a)
                os.replace(tmp, os.path.join(d, f + ".npy"))
    return g


def random_csr(n_rows: int, n_cols: int, rng: np.random.Generator, mean_deg: float = 4.0,
               max_deg: int | None = None, dup: bool = False, unsorted: bool = False,
               empty_frac: float = 0.0, values: bool = True) -> Graph:
    """Small irregular test graph: geometric-ish degrees, optional empty rows,
    duplicate (i, j) pairs and unsorted columns."""
    deg = rng.geometric(1.0 / (mean_deg + 1.0), size=n_rows) - 1
    if max_deg is not None:
        deg = np.minimum(deg, max_deg)
    if empty_frac > 0:
        deg[rng.random(n_rows) < empty_frac] = 0
    if not dup:
        deg = np.minimum(deg, n_cols)
    rowptr = np.zeros(n_rows + 1, dtype=np.int64)
    np.cumsum(deg, out=rowptr[1:])
    cols = []
    for i in range(n_rows):
        if deg[i] == 0:
            continue
        if dup:
            c = rng.integers(0, n_cols, size=deg[i])
        else:
            c = rng.choice(n_cols, size=deg[i], replace=False)
        if not unsorted:
            c = np.sort(c)
        cols.append(c)
    col = np.concatenate(cols).astype(np.int32) if cols else np.zeros(0, np.int32)
    val = rng.standard_normal(col.size).astype(np.float32) if values else None
    return Graph(rowptr.astype(np.int32), col, val, n_rows, n_cols)


# ------------------------------------------------ 2-layer inference workload

# The end-to-end inference workload (2-layer GCN and GAT, hidden size 128, the
# GAT with 4 heads) on the Reddit-shaped dense-degree graph of workload 3,
# with Reddit's feature and class counts (602 inputs, 41 classes).
INFERENCE = dict(graph=3, F_in=602, hidden=128, classes=41, heads=4, head_dim=32, slope=0.2)


def model_params(kind: str, F_in: int, hidden: int, classes: int, heads: int = 1, seed: int = 7000):
    """Seeded fp32 parameters of a 2-layer model (Glorot-like scales; biases small):
    GCN: W1 [hidden, F_in], b1, W2 [classes, hidden], b2.
    GAT: W1 [hidden, F_in] (hidden = heads * head dim), a_src1 / a_dst1 [heads, hidden/heads],
    b1 [hidden], W2 [classes, hidden], a_src2 / a_dst2 [1, classes], b2 [classes]."""
    rng = np.random.default_rng(seed)
    f32 = np.float32
    p = dict(W1=(rng.standard_normal((hidden, F_in)) / np.sqrt(F_in)).astype(f32),
             b1=(0.1 * rng.standard_normal(hidden)).astype(f32),
             W2=(rng.standard_normal((classes, hidden)) / np.sqrt(hidden)).astype(f32),
             b2=(0.1 * rng.standard_normal(classes)).astype(f32))
    if kind == "gat":
        D = hidden // heads
        p["a_src1"] = (rng.standard_normal((heads, D)) / np.sqrt(D)).astype(f32)
        p["a_dst1"] = (rng.standard_normal((heads, D)) / np.sqrt(D)).astype(f32)
        p["a_src2"] = (rng.standard_normal((1, classes)) / np.sqrt(classes)).astype(f32)
        p["a_dst2"] = (rng.standard_normal((1, classes)) / np.sqrt(classes)).astype(f32)
    return p
