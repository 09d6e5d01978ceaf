"""Column-sliced plans (cogdl_plan_create_sliced): the work units against their
definition (each row cut into contiguous pieces, a long row of sorted columns
at the boundaries of 8 equal column ranges, pieces of at most group_size
edges), and every plan-driven operator with a sliced plan against the oracle:
SpMM, mean and max (edge ids bit for bit), SpMM^T on a plan sliced by the
CSC's rows, the GAT aggregation and softmax, SDDMM and the GAT backward with
sliced CSR and CSC plans.  Graphs come from the seeded random sweep, with
slice thresholds low enough that most rows are sliced."""
import numpy as np
import pytest

import oracle

from gpu_util import TOL_ALPHA, TOL_F32, dev, features, graph_to_dev, say, scaled_error, to_f64, tol_for
from test_gpu_random import KINDS, _case, _close

pytestmark = pytest.mark.gpu

N_CASES = 100
SLICES = 8


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _spec(seed):
    rng = np.random.default_rng(7700 + seed)
    G = int(rng.choice([0, 2, 5, 16, 64]))
    slice_min = int(rng.choice([1, 3, 8, 40]))
    mode = ["auto", "neighbor_group", "row_split"][int(rng.integers(0, 3))]
    return mode, G, slice_min


def _sliced(cg, rp, cl, nnz, n_cols, spec, max_feat, max_heads=0):
    mode, G, smin = spec
    return cg.Plan(rp, nnz, max_feat=max_feat, max_heads=max_heads, mode=mode, group_size=G,
                   col=cl, n_cols=n_cols, slice_min=smin)


def expected_pieces(rowptr, col, n_cols, G, smin, ng):
    """The definition: per row, its contiguous pieces (begin, end)."""
    width = max(1, -(-n_cols // SLICES))
    out = []
    for i in range(len(rowptr) - 1):
        b, e = int(rowptr[i]), int(rowptr[i + 1])
        d = e - b
        if not ng:
            out.append((i, b, e))
            continue
        if d > smin:
            # lower bound of each boundary column over the whole row, then a running
            # maximum (the exact boundaries on sorted rows, ordered cuts on any row)
            cuts = [b]
            for s in range(1, SLICES):
                lo, hi = b, e
                while lo < hi:
                    mid = (lo + hi) // 2
                    if col[mid] < s * width:
                        lo = mid + 1
                    else:
                        hi = mid
                cuts.append(max(lo, cuts[-1]))
            cuts.append(e)
        else:
            cuts = [b, e]
        if d == 0:
            out.append((i, b, e))
            continue
        for s in range(len(cuts) - 1):
            for p in range(cuts[s], cuts[s + 1], G):
                out.append((i, p, min(p + G, cuts[s + 1])))
    return sorted(out)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sliced_units_match_definition(cg, seed):
    rng, g, _ = _case(seed)
    mode, G, smin = _spec(seed)
    rp, cl, _ = graph_to_dev(g)
    plan = _sliced(cg, rp, cl, g.nnz, g.n_cols, (mode, G, smin), 8)
    try:
        info = plan.info()
        units = plan.units().cpu().numpy()
        ng = info["mode"] == 2
        want = expected_pieces(g.rowptr, g.col, g.n_cols, info["group_size"], smin, ng)
        assert sorted(map(tuple, units[:, :3].tolist())) == want
        # partial slots exactly on the rows cut into several pieces, numbered densely
        per_row = np.bincount(units[:, 0], minlength=g.n_rows)
        split = units[:, 3] >= 0
        assert np.array_equal(split, per_row[units[:, 0]] > 1)
        if split.any():
            assert np.array_equal(np.sort(units[split, 3]), np.arange(split.sum()))
        assert info["n_partials"] == split.sum()
        # a sliced row of sorted columns: every piece inside one column range
        width = max(1, -(-g.n_cols // SLICES))
        for r, b, e, _ in units:
            if ng and e - b > 0 and g.rowptr[r + 1] - g.rowptr[r] > smin:
                cols = g.col[b:e]
                if np.all(np.diff(g.col[g.rowptr[r]:g.rowptr[r + 1]]) >= 0):
                    assert cols.min() // width == cols.max() // width
        # rebuilding gives the same units; a plain rebuild is refused
        u0 = plan.units().clone()
        plan.rebuild(rp, cl)
        import torch
        assert torch.equal(u0, plan.units())
        with pytest.raises(cg.CogdlError):
            cg._check(cg.lib().cogdl_plan_rebuild(plan.handle, cg._ptr(rp), cg._stream()), "rebuild")
    finally:
        plan.close()


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sliced_spmm_family(cg, seed):
    import torch
    rng, g, _ = _case(seed)
    spec = _spec(seed)
    F = int(rng.choice([1, 3, 8, 16, 64, 100, 256]))
    xk = KINDS[int(rng.integers(0, 3))]
    say(f"sliced spmm {seed}: {g.n_rows}x{g.n_cols} nnz={g.nnz} F={F} {xk} plan={spec}")
    rp, cl, vl = graph_to_dev(g)
    xh, xc, xd = features((g.n_cols, F), 300 + seed, xk)
    plan = _sliced(cg, rp, cl, g.nnz, g.n_cols, spec, F)
    try:
        Y = cg.spmm(rp, cl, vl, xd, plan=plan, out_dtype=torch.float32)
        Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh, x_dtype=xc)
        assert scaled_error(Y, Yr, Ar) <= tol_for(xk, "f32"), "spmm"
        Ym = cg.gspmm(rp, cl, vl, xd, "mean", plan=plan, out_dtype=torch.float32)
        Ymr, Amr, _ = oracle.gspmm(g.rowptr, g.col, g.val, xh, "mean", n_cols=g.n_cols, x_dtype=xc)
        assert scaled_error(Ym, Ymr, Amr) <= tol_for(xk, "f32"), "mean"
        Yx, arg = cg.gspmm(rp, cl, vl, xd, "max", plan=plan, out_dtype=torch.float32, return_arg=True)
        Yxr, _, ar = oracle.gspmm(g.rowptr, g.col, g.val, xh, "max", n_cols=g.n_cols, x_dtype=xc)
        want = oracle.decode(oracle.round_to(Yxr, oracle.F32), oracle.F32)
        assert np.array_equal(to_f64(Yx).reshape(Yxr.shape), want.reshape(Yxr.shape)), "max"
        assert np.array_equal(arg.cpu().numpy().reshape(ar.shape), ar), "argmax"
    finally:
        _close(plan)
    colptr, row_t, val_t, _ = cg.csr_to_csc(rp, cl, vl, g.n_cols)
    gh, gc, gd = features((g.n_rows, F), 400 + seed, xk)
    plan_t = _sliced(cg, colptr, row_t, g.nnz, g.n_rows, spec, F)
    try:
        dX = cg.spmm_t(colptr, row_t, val_t, gd, plan_t=plan_t, out_dtype=torch.float32)
        dXr, dAr = oracle.spmm_t(g.rowptr, g.col, g.val, gh, g.n_cols, g_dtype=gc)
        assert scaled_error(dX, dXr, dAr) <= tol_for(xk, "f32"), "spmm_t"
    finally:
        _close(plan_t)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_sliced_gat_forward_backward(cg, seed):
    import torch
    rng, g, _ = _case(seed)
    spec = _spec(seed)
    H = int(rng.choice([1, 2, 4, 8]))
    D = int(rng.choice([1, 4, 16, 32, 64]))
    xk = ["f32", "bf16"][int(rng.integers(0, 2))]
    say(f"sliced gat {seed}: {g.n_rows}x{g.n_cols} nnz={g.nnz} H={H} D={D} {xk} plan={spec}")
    rp, cl, _ = graph_to_dev(g)
    srng = np.random.default_rng(500 + seed)
    sd = srng.standard_normal((g.n_rows, H)).astype(np.float32)
    ss = srng.standard_normal((g.n_cols, H)).astype(np.float32)
    xh, xc, xd = features((g.n_cols, H, D), 600 + seed, xk)
    a_ref = oracle.edge_softmax(g.rowptr, g.col, sd, ss, slope=0.2)
    plan = _sliced(cg, rp, cl, g.nnz, g.n_cols, spec, H * D, max_heads=H)
    try:
        Y, a = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xd, 0.2, plan=plan, out_dtype=torch.float32,
                                return_alpha=True)
        Yr, Ar = oracle.gat(g.rowptr, g.col, sd, ss, xh.reshape(g.n_cols, H * D), H, D, slope=0.2, x_dtype=xc)
        assert scaled_error(Y.reshape(g.n_rows, H * D), Yr, Ar) <= tol_for(xk, "f32"), "gat"
        a_s = cg.sddmm_edge_softmax(rp, cl, dev(sd), dev(ss), 0.2, plan=plan)
        if g.nnz:
            for got, what in ((a, "alpha"), (a_s, "softmax")):
                rel = np.abs(to_f64(got).reshape(a_ref.shape) - a_ref) / a_ref
                assert rel.max() <= TOL_ALPHA, what
        pq = features((g.n_rows, H, D), 650 + seed, xk)
        S = cg.sddmm_dot(rp, cl, pq[2], xd, plan=plan)
        Sr, Sa = oracle.sddmm_dot(g.rowptr, g.col, pq[0].reshape(g.n_rows, H * D), xh.reshape(g.n_cols, H * D),
                                  H, D, p_dtype=pq[1], q_dtype=xc)
        assert scaled_error(S.reshape(Sr.shape), Sr, Sa) <= TOL_F32, "sddmm"
    finally:
        _close(plan)
    alpha = a_ref.astype(np.float32)
    gh, gc, gd = features((g.n_rows, H, D), 700 + seed, xk)
    colptr, row_t, _, perm = oracle.csr_to_csc(g.rowptr, g.col, None, g.n_cols)
    cp_d, rt_d, pm_d = dev(colptr), dev(row_t), dev(perm)
    ref = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, xh.reshape(g.n_cols, H * D),
                              gh.reshape(g.n_rows, H * D), H, D, slope=0.2, x_dtype=xc, dy_dtype=gc)
    plan = _sliced(cg, rp, cl, g.nnz, g.n_cols, spec, H * D, max_heads=H)
    plan_t = _sliced(cg, cp_d, rt_d, g.nnz, g.n_rows, spec, H * D, max_heads=H)
    try:
        out = cg.gat_backward(rp, cl, cp_d, rt_d, pm_d, dev(sd), dev(ss), dev(alpha), xd, gd, 0.2,
                              plan=plan, plan_t=plan_t, dx_dtype=torch.float32)
        for k in ("dalpha", "dscore", "ds_dst", "ds_src"):
            assert scaled_error(out[k], ref[k], ref[k + "_abs"]) <= TOL_F32, k
        assert scaled_error(out["dX"].reshape(ref["dX"].shape), ref["dX"], ref["dX_abs"]) <= TOL_F32, "dX"
    finally:
        _close(plan, plan_t)


def _degree_graph(deg, n_cols, seed):
    rng = np.random.default_rng(seed)
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
    col = np.concatenate([np.sort(rng.choice(n_cols, d, replace=False)) for d in deg]).astype(np.int32)
    from paper_2103_00959_amd import synth
    return synth.Graph(rowptr, col, rng.standard_normal(col.size).astype(np.float32), len(deg), n_cols)


def test_sliced_rebuild_beyond_capacity_falls_back(cg):
    """A sliced plan sized on one graph, rebuilt on a graph with the same n_rows and nnz but
    far more sliced units than it has room for: that build slices no row (the plain
    neighbour groups, unit for unit) and every result stays right; rebuilt on the first graph
    again, it slices as before."""
    import torch
    n, n_cols, smin = 1000, 1000, 32
    deg_a = np.full(n, 6, np.int64)
    deg_a[7] = 206                                  # one row over the slice threshold
    deg_b = np.full(n, 1, np.int64)
    deg_b[:20] = 250                                # twenty long rows, 8 pieces each
    deg_b[20:] = (deg_a.sum() - 20 * 250) // (n - 20)
    deg_b[-1] += deg_a.sum() - deg_b.sum()
    assert deg_a.sum() == deg_b.sum()
    ga, gb = _degree_graph(deg_a, n_cols, 1), _degree_graph(deg_b, n_cols, 2)
    E = int(deg_a.sum())
    rpa, cla, vla = graph_to_dev(ga)
    rpb, clb, vlb = graph_to_dev(gb)
    plan = cg.Plan(rpa, E, max_feat=64, mode="neighbor_group", col=cla, n_cols=n_cols, slice_min=smin)
    try:
        info = plan.info()
        G = info["group_size"]
        units_a = sorted(map(tuple, plan.units().cpu().numpy()[:, :3].tolist()))
        assert units_a == expected_pieces(ga.rowptr, ga.col, n_cols, G, smin, True)
        for g, rp, cl, vl, sliced in ((gb, rpb, clb, vlb, False), (ga, rpa, cla, vla, True)):
            plan.rebuild(rp, cl)
            units = sorted(map(tuple, plan.units().cpu().numpy()[:, :3].tolist()))
            if sliced:
                assert units == units_a
            else:
                plain = sorted(map(tuple, oracle.neighbor_groups(g.rowptr, G, 2).tolist()))
                assert units == plain
                assert len(expected_pieces(g.rowptr, g.col, n_cols, G, smin, True)) > plan.info()["n_units"]
            xh, xc, xd = features((n_cols, 64), 5, "f32")
            Y = cg.spmm(rp, cl, vl, xd, plan=plan)
            Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh, x_dtype=xc)
            assert scaled_error(Y, Yr, Ar) <= TOL_F32
            torch.cuda.synchronize()
    finally:
        plan.close()
