"""GPU parity at the workloads' full sizes.

The medium R-MAT workload (169,343 nodes, 2.5M nonzeros) is compared element
by element.  The large workloads (114.6M, 64.3M and 122.4M nonzeros) run in the
launch configuration the benchmark times (balancer on AUTO, default group
size, the benchmark's dtypes) and are compared on sampled rows (or columns)
that the oracle computes one by one: a seeded random sample plus the rows with
the largest degrees, where split rows and long fp32 sums live.  Integer
outputs (the transpose, the balancer's mode) are compared in full.
"""
import numpy as np
import pytest

import oracle
from paper_2103_00959_amd import synth

from gpu_util import (TOL_16, TOL_ALPHA, TOL_F32, alpha_bound_scale, alpha_close, dev, features, say,
                      scaled_error)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _sample_rows(g, n_random=1500, n_top=12, seed=123):
    d = g.degrees()
    top = np.argsort(-d, kind="stable")[:n_top]
    rnd = np.random.default_rng(seed).choice(g.n_rows, size=min(n_random, g.n_rows), replace=False)
    return np.unique(np.concatenate([top, rnd])).astype(np.int32)


def _edges_of(g, rows):
    return np.concatenate([np.arange(g.rowptr[r], g.rowptr[r + 1]) for r in rows])


@pytest.mark.timeout(900)
def test_medium_rmat_full(cg):
    """169,343 nodes, 2.5M nonzeros, F = 128 fp32: every output element."""
    import torch
    g = synth.config_graph(2, verbose=True)
    say(f"medium R-MAT n={g.n_rows} nnz={g.nnz}")
    rp, cl, vl = dev(g.rowptr), dev(g.col), dev(g.val)
    xh, xc, xd = features((g.n_cols, 128), 2002, "f32")
    plan = cg.Plan(rp, g.nnz, 128)
    try:
        assert plan.info()["mode"] == oracle.balance_mode(g.rowptr, g.nnz)
        Y = cg.spmm(rp, cl, vl, xd, plan=plan)
        Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh)
        assert scaled_error(Y, Yr, Ar) <= TOL_F32
    finally:
        plan.close()
    colptr, row_t, val_t, perm = cg.csr_to_csc(rp, cl, vl, g.n_cols)
    c_ref, r_ref, v_ref, p_ref = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
    assert np.array_equal(colptr.cpu().numpy(), c_ref)
    assert np.array_equal(perm.cpu().numpy(), p_ref)
    assert np.array_equal(row_t.cpu().numpy(), r_ref)
    assert np.array_equal(val_t.cpu().numpy().view(np.uint32), v_ref.view(np.uint32))
    gh, gc, gd = features((g.n_rows, 128), 4002, "f32")
    plan_t = cg.Plan(colptr, g.nnz, 128)
    try:
        dX = cg.spmm_t(colptr, row_t, val_t, gd, plan_t=plan_t)
        dXr, dAr = oracle.spmm_t(g.rowptr, g.col, g.val, gh, g.n_cols)
        assert scaled_error(dX, dXr, dAr) <= TOL_F32
    finally:
        plan_t.close()
    torch.cuda.synchronize()


@pytest.mark.timeout(900)
def test_dense_degree_sampled(cg):
    """232,965 nodes, 114.6M nonzeros (mean degree 492, max 20k), F = 256 fp32."""
    g = synth.config_graph(3, verbose=True)
    say(f"dense-degree n={g.n_rows} nnz={g.nnz}")
    rp, cl, vl = dev(g.rowptr), dev(g.col), dev(g.val)
    xh, xc, xd = features((g.n_cols, 256), 2003, "f32")
    plan = cg.Plan(rp, g.nnz, 256)
    try:
        assert plan.info()["mode"] == oracle.balance_mode(g.rowptr, g.nnz)
        Y = cg.spmm(rp, cl, vl, xd, plan=plan)
        rows = _sample_rows(g)
        Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh, rows=rows)
        import torch
        err = scaled_error(Y[torch.from_numpy(rows).long().cuda()], Yr, Ar)
        say(f"dense-degree sampled error {err:.3g}")
        assert err <= TOL_F32
        # row-normalized weights: every row of A 1 is 1 (a property at any size)
        ones = torch.ones((g.n_cols, 4), dtype=torch.float32, device="cuda")
        Y1 = cg.spmm(rp, cl, vl, ones, plan=plan)
        d = torch.from_numpy(g.degrees()).cuda().float()
        assert float(((Y1[:, 0] - 1.0).abs() / (d * 2.0 ** -23 + 2.0 ** -23)).max()) <= 4.0
    finally:
        plan.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("sliced", [True, False])
def test_gat_layer_sampled(cg, sliced):
    """2,449,029 nodes, 64.3M nonzeros, H = 8 x D = 16 fp32, alpha written; with the
    column-sliced plan the workload's benchmark line builds (split rows: the alpha of their
    neighbour groups takes the split-row pass), and with a plain one."""
    import torch
    g = synth.config_graph(4, verbose=True)
    H, D = 8, 16
    say(f"GAT layer n={g.n_rows} nnz={g.nnz} sliced={sliced}")
    rp, cl = dev(g.rowptr), dev(g.col)
    rng = np.random.default_rng(3004)
    sd = rng.standard_normal((g.n_rows, H), dtype=np.float32)
    ss = rng.standard_normal((g.n_cols, H), dtype=np.float32)
    xh, xc, xd = features((g.n_cols, H, D), 2004, "f32")
    plan = cg.Plan(rp, g.nnz, H * D, max_heads=H, **(dict(col=cl, n_cols=g.n_cols) if sliced else {}))
    try:
        Y, alpha = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xd, 0.2, plan=plan, return_alpha=True)
        a2 = cg.sddmm_edge_softmax(rp, cl, dev(sd), dev(ss), 0.2, plan=plan)
        rows = _sample_rows(g)
        Yr, Ar = oracle.gat(g.rowptr, g.col, sd, ss, xh.reshape(g.n_cols, H * D), H, D, slope=0.2,
                            rows=rows)
        idx = torch.from_numpy(rows).long().cuda()
        err = scaled_error(Y.reshape(g.n_rows, H * D)[idx], Yr, Ar)
        say(f"GAT sampled error {err:.3g}")
        assert err <= TOL_F32
        if sliced:
            assert plan.info()["n_split_rows"] > 0    # the split-row alpha pass is exercised
        a_ref = oracle.edge_softmax(g.rowptr, g.col, sd, ss, slope=0.2, rows=rows)
        e_idx = torch.from_numpy(_edges_of(g, rows)).long().cuda()
        bound = alpha_bound_scale(g.rowptr, g.col, sd, ss, rows=rows)
        for a in (alpha, a2):
            err = alpha_close(a[e_idx], a_ref, bound)
            say(f"GAT alpha sampled error {err:.3g} x bound")
            assert err <= TOL_ALPHA
    finally:
        plan.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("sliced", [True, False])
def test_skewed_mixed_precision_sampled(cg, sliced):
    """2.4M nodes, 122.4M nonzeros with 100k-300k-edge hubs, bf16 features:
    the benchmark's launch configuration (SpMM, transpose, SpMM^T, fused GAT;
    column-sliced plans as the benchmark builds them, and plain ones)."""
    import torch
    g = synth.config_graph(5, verbose=True)
    N, E = g.n_rows, g.nnz
    F, H, D = 256, 4, 64
    say(f"skewed n={N} nnz={E}")
    rp, cl, vl = dev(g.rowptr), dev(g.col), dev(g.val)
    xh, xc, xd = features((N, F), 2005, "bf16")
    plan = cg.Plan(rp, E, max_feat=F, max_heads=H, **(dict(col=cl, n_cols=N) if sliced else {}))
    rows = _sample_rows(g)
    idx = torch.from_numpy(rows).long().cuda()
    try:
        info = plan.info()
        assert info["mode"] == oracle.balance_mode(g.rowptr, E)
        Y = cg.spmm(rp, cl, vl, xd, plan=plan)
        Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh, x_dtype=xc, rows=rows)
        err = scaled_error(Y[idx], Yr, Ar)
        say(f"skewed SpMM sampled error {err:.3g}")
        assert err <= TOL_16
        # the fp32-output error stays at the fp32 level even on the hub rows
        Y32 = cg.spmm(rp, cl, vl, xd, plan=plan, out_dtype=torch.float32)
        assert scaled_error(Y32[idx], Yr, Ar) <= TOL_F32
        # GAT 4 x 64 bf16
        rng = np.random.default_rng(3005)
        sd = rng.standard_normal((N, H), dtype=np.float32)
        ss = rng.standard_normal((N, H), dtype=np.float32)
        xgh, xgc, xgd = features((N, H, D), 2105, "bf16")
        Yg = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xgd, 0.2, plan=plan,
                              out_dtype=torch.float32)
        Ygr, Agr = oracle.gat(g.rowptr, g.col, sd, ss, xgh.reshape(N, H * D), H, D, slope=0.2,
                              x_dtype=xgc, rows=rows)
        err = scaled_error(Yg.reshape(N, H * D)[idx], Ygr, Agr)
        say(f"skewed GAT sampled error {err:.3g}")
        assert err <= TOL_F32
        # the benchmark's output dtype: bf16 rows
        Yb = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xgd, 0.2, plan=plan)
        assert Yb.dtype == torch.bfloat16
        err = scaled_error(Yb.reshape(N, H * D)[idx], Ygr, Agr)
        say(f"skewed GAT bf16-out sampled error {err:.3g}")
        assert err <= TOL_16
        del Yb, Yg
        # the benchmark's step: source scores projected from the gathered rows
        # (s_src = X a_src, a_src N(0, 1/D)), bf16 out; the oracle's fp64 head scores feed its
        # aggregation, and the bar adds the score's own rounding (as for the small graphs)
        a_src = (np.random.default_rng(3105).standard_normal((H, D)) / np.sqrt(D)).astype(np.float32)
        Yp = cg.gat_aggregate_proj(rp, cl, dev(sd), dev(a_src), xgd, 0.2, plan=plan)
        assert Yp.dtype == torch.bfloat16
        ss_ref, _, ss_abs, _ = oracle.head_scores(xgh.reshape(N, H * D), a_src, a_src, H, D, z_dtype=xgc)
        Ypr, Apr = oracle.gat(g.rowptr, g.col, sd, ss_ref.astype(np.float32), xgh.reshape(N, H * D), H, D,
                              slope=0.2, x_dtype=xgc, rows=rows)
        u = 2.0 ** -24
        score_term = 2 * (D * u * float(ss_abs.max()) + u * float(np.abs(ss_ref).max()))
        err = scaled_error(Yp.reshape(N, H * D)[idx], Ypr, Apr)
        say(f"skewed projected GAT bf16-out sampled error {err:.3g} (score term {score_term:.2g})")
        assert err <= TOL_16 + score_term
        del Yp, ss_ref, ss_abs
    finally:
        plan.close()
    # transpose: bit-exact in full
    colptr, row_t, val_t, perm = cg.csr_to_csc(rp, cl, vl, N)
    c_ref, r_ref, v_ref, p_ref = oracle.csr_to_csc(g.rowptr, g.col, g.val, N)
    assert np.array_equal(colptr.cpu().numpy(), c_ref)
    assert np.array_equal(perm.cpu().numpy(), p_ref)
    assert np.array_equal(row_t.cpu().numpy(), r_ref)
    assert np.array_equal(val_t.cpu().numpy().view(np.uint32), v_ref.view(np.uint32))
    del c_ref, r_ref, v_ref, p_ref
    gh, gc, gd = features((N, F), 4005, "bf16")
    plan_t = cg.Plan(colptr, E, max_feat=F, **(dict(col=row_t, n_cols=N) if sliced else {}))
    try:
        dX = cg.spmm_t(colptr, row_t, val_t, gd, plan_t=plan_t, out_dtype=torch.float32)
        cdeg = np.diff(c_ref_cols := colptr.cpu().numpy())
        top = np.argsort(-cdeg, kind="stable")[:12]
        cols = np.unique(np.concatenate([top, np.random.default_rng(7).choice(N, 1500, replace=False)]))
        cols = cols.astype(np.int32)
        dXr, dAr = oracle.spmm_t(g.rowptr, g.col, g.val, gh, N, g_dtype=gc, cols=cols)
        err = scaled_error(dX[torch.from_numpy(cols).long().cuda()], dXr, dAr)
        say(f"skewed SpMM^T sampled error {err:.3g}")
        assert err <= TOL_F32
        del c_ref_cols
    finally:
        plan_t.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("sliced", [True, False])
def test_gat_backward_skewed_sampled(cg, sliced):
    """2.4M nodes, 122.4M nonzeros with hubs, H = 4 x D = 64 bf16: the GAT
    backward in the benchmark's launch configuration, compared on sampled rows
    (attention and score gradients, ds_dst) and sampled columns (ds_src, dX),
    the largest in-degree columns included."""
    import torch
    g = synth.config_graph(5, verbose=True)
    N, E = g.n_rows, g.nnz
    H, D = 4, 64
    say(f"GAT backward skewed n={N} nnz={E}")
    rp, cl = dev(g.rowptr), dev(g.col)
    rng = np.random.default_rng(3105)
    sd = rng.standard_normal((N, H), dtype=np.float32)
    ss = rng.standard_normal((N, H), dtype=np.float32)
    alpha = rng.random((E, H), dtype=np.float32)
    xh, xc, xd = features((N, H, D), 2205, "bf16")
    gh, gc, gd = features((N, H, D), 4105, "bf16")
    colptr, row_t, _, perm = cg.csr_to_csc(rp, cl, None, N)
    plan = cg.Plan(rp, E, max_feat=H * D, max_heads=H, **(dict(col=cl, n_cols=N) if sliced else {}))
    plan_t = cg.Plan(colptr, E, max_feat=H * D, max_heads=H, **(dict(col=row_t, n_cols=N) if sliced else {}))
    try:
        out = cg.gat_backward(rp, cl, colptr, row_t, perm, dev(sd), dev(ss), dev(alpha), xd, gd, 0.2,
                              plan=plan, plan_t=plan_t)
        torch.cuda.synchronize()
    finally:
        plan.close()
        plan_t.close()
    rows = _sample_rows(g)
    cdeg = np.diff(colptr.cpu().numpy())
    cols = np.unique(np.concatenate([np.argsort(-cdeg, kind="stable")[:12],
                                     np.random.default_rng(8).choice(N, 1500, replace=False)])).astype(np.int32)
    ref = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, xh.reshape(N, H * D), gh.reshape(N, H * D),
                              H, D, slope=0.2, x_dtype=xc, dy_dtype=gc, rows=rows, cols=cols)
    e_idx = torch.from_numpy(_edges_of(g, rows)).long().cuda()
    r_idx = torch.from_numpy(rows).long().cuda()
    c_idx = torch.from_numpy(cols).long().cuda()
    for k, got in (("dalpha", out["dalpha"][e_idx]), ("dscore", out["dscore"][e_idx]),
                   ("ds_dst", out["ds_dst"][r_idx]), ("ds_src", out["ds_src"][c_idx])):
        err = scaled_error(got, ref[k], ref[k + "_abs"])
        say(f"GAT backward {k} sampled error {err:.3g}")
        assert err <= TOL_F32, k
    err = scaled_error(out["dX"].reshape(N, H * D)[c_idx], ref["dX"], ref["dX_abs"])
    say(f"GAT backward dX sampled error {err:.3g}")
    assert err <= TOL_16


@pytest.mark.timeout(900)
def test_gat_training_pair_skewed(cg):
    """The training pair at full size (2.4M nodes, 122.4M nonzeros, 4 x 64 bf16, the benchmark's
    sliced plans): the forward that keeps each row's softmax state gives the alpha-writing
    forward's Y bit for bit, and the backward that rebuilds the weights from those states gives
    the backward on that alpha bit for bit (the layer gradients and the (alpha, dscore) records,
    whose weights are the forward's alpha)."""
    import torch
    g = synth.config_graph(5, verbose=True)
    N, E = g.n_rows, g.nnz
    H, D = 4, 64
    say(f"GAT training pair skewed n={N} nnz={E}")
    rp, cl = dev(g.rowptr), dev(g.col)
    rng = np.random.default_rng(3107)
    sd = dev(rng.standard_normal((N, H), dtype=np.float32))
    ss = dev(rng.standard_normal((N, H), dtype=np.float32))
    _, _, xd = features((N, H, D), 2207, "bf16")
    _, _, gd = features((N, H, D), 4107, "bf16")
    colptr, row_t, _, perm = cg.csr_to_csc(rp, cl, None, N)
    plan = cg.Plan(rp, E, max_feat=H * D, max_heads=H, col=cl, n_cols=N)
    plan_t = cg.Plan(colptr, E, max_feat=H * D, max_heads=H, col=row_t, n_cols=N)
    try:
        Ya, alpha = cg.gat_aggregate(rp, cl, sd, ss, xd, 0.2, plan=plan, return_alpha=True)
        Ys, st = cg.gat_aggregate_stats(rp, cl, sd, xd, s_src=ss, plan=plan)
        assert torch.equal(Ya, Ys)
        del Ya, Ys
        o = {"dalpha": None, "dscore": None}
        ba = cg.gat_backward(rp, cl, colptr, row_t, perm, sd, ss, alpha, xd, gd, 0.2, plan=plan,
                             plan_t=plan_t, out=dict(o))
        bs = cg.gat_backward(rp, cl, colptr, row_t, perm, sd, ss, None, xd, gd, 0.2, plan=plan,
                             plan_t=plan_t, out=dict(o), row_stats=st)
        torch.cuda.synchronize()
        for k in ("dX", "ds_dst", "ds_src", "edge_work"):
            assert torch.equal(ba[k], bs[k]), k
        assert torch.equal(bs["edge_work"][..., 0].reshape(-1), alpha.reshape(-1))
        say("GAT training pair skewed: bit for bit")
    finally:
        plan.close()
        plan_t.close()


@pytest.mark.timeout(900)
def test_inference_reddit_shaped_sampled(cg):
    """2-layer GCN and GAT inference (hidden 128, 4 heads, 602 inputs, 41 classes) on
    the Reddit-shaped graph (232,965 nodes, 114.6M nonzeros), bf16 activations:
    sampled output rows against the oracle models, within the model bound."""
    import torch
    spec = synth.INFERENCE
    g = synth.config_graph(spec["graph"], verbose=True)
    N = g.n_rows
    k, hid, C, Hh = spec["F_in"], spec["hidden"], spec["classes"], spec["heads"]
    rp, cl, vl = dev(g.rowptr), dev(g.col), dev(g.val)
    xb = synth.f32_to_bf16_bits(synth.normal_f32((N, k), 7003))
    xd = dev(xb.view(np.int16)).view(torch.bfloat16)
    rows = _sample_rows(g, n_random=800)
    idx = torch.from_numpy(rows).long().cuda()
    plan = cg.Plan(rp, g.nnz, max_feat=hid, max_heads=Hh)
    try:
        for kind in ("gcn", "gat"):
            p = synth.model_params(kind, k, hid, C, Hh, seed=7100 if kind == "gcn" else 7200)
            host = {n: (synth.f32_to_bf16_bits(v) if n.startswith("W") else v) for n, v in p.items()}
            devp = {n: (dev(synth.f32_to_bf16_bits(v).view(np.int16)).view(torch.bfloat16)
                        if n.startswith("W") else dev(v)) for n, v in p.items()}
            if kind == "gcn":
                Y = cg.gcn_forward(rp, cl, vl, xd, devp, plan=plan)
                Yr, E = oracle.gcn_forward(g.rowptr, g.col, g.val, xb, host, rows=rows)
            else:
                Y = cg.gat_forward(rp, cl, xd, devp, spec["slope"], plan=plan)
                Yr, E = oracle.gat_forward(g.rowptr, g.col, xb, host, slope=spec["slope"], rows=rows)
            err = scaled_error(Y[idx], Yr, E)
            say(f"{kind} inference sampled error {err:.3g}")
            assert err <= 3 * 2.0 ** -7 + 1e-3, kind
    finally:
        plan.close()


@pytest.mark.timeout(900)
def test_features_beyond_4gib_use_64bit_gathers(cg):
    """A feature matrix larger than the 32-bit offsets of the buffer gathers reach
    (1,100,000 x 2048 bf16 = 4.2 GiB) takes the 64-bit gather path: the SpMM and
    the GAT aggregation gather rows near its end, whole rows and split rows."""
    import torch
    n_cols, W = 1_100_000, 2048
    rng = np.random.default_rng(77)
    n_rows = 3000
    deg = rng.integers(0, 40, n_rows)
    deg[[0, 17, 2999]] = [5000, 3000, 1]                  # split rows under a small group size
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
    col = np.concatenate([np.sort(rng.choice(n_cols, d, replace=False)) for d in deg]).astype(np.int32)
    col[::7] = n_cols - 1 - (np.arange(col[::7].size) % 5)  # rows at the very end of X
    val = rng.standard_normal(col.size).astype(np.float32)
    say(f"huge X: {n_cols} x {W} bf16 = {n_cols * W * 2 / 2**30:.2f} GiB, nnz={col.size}")
    xb = synth.f32_to_bf16_bits(synth.normal_f32((n_cols, W), 9001))
    xd = dev(xb.view(np.int16)).view(torch.bfloat16)
    rp, cl, vl = dev(rowptr), dev(col), dev(val)
    rows = np.unique(np.concatenate([[0, 17, 2999], rng.choice(n_rows, 200, replace=False)])).astype(np.int32)
    idx = torch.from_numpy(rows).long().cuda()
    for spec in (None, ("neighbor_group", 256)):
        plan = None if spec is None else cg.Plan(rp, col.size, W, max_heads=8, mode=spec[0], group_size=spec[1])
        try:
            Y = cg.spmm(rp, cl, vl, xd, plan=plan, out_dtype=torch.float32)
            Yr, Ar = oracle.spmm(rowptr, col, val, xb, x_dtype=oracle.BF16, rows=rows)
            assert scaled_error(Y[idx], Yr, Ar) <= TOL_F32, spec
            H, D = 8, W // 8
            alpha = rng.random((col.size, H)).astype(np.float32)
            Yg = cg.gat_aggregate(rp, cl, None, None, xd.view(n_cols, H, D), alpha_in=dev(alpha), plan=plan,
                                  out_dtype=torch.float32)
            Ygr, Agr = oracle.gat(rowptr, col, None, None, xb, H, D, alpha_in=alpha, x_dtype=oracle.BF16,
                                  rows=rows)
            assert scaled_error(Yg.reshape(n_rows, W)[idx], Ygr, Agr) <= TOL_F32, spec
        finally:
            if plan is not None:
                plan.close()
    del xd
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_max_nnz_int32_edge_ids(cg):
    """The largest edge count the int32 edge ids allow (2^31 - 4097 nonzeros, 8.6 GB per
    edge array): the SpMM on sampled rows and SpMM^T on sampled columns against the oracle,
    the transpose checked on every slot by its definition (column counts, each slot's column,
    row and value bits, edge ids increasing inside a column, which together make perm a
    permutation)."""
    import torch
    nnz = cg.MAX_NNZ
    n_rows, n_cols, F = 1 << 20, 4093, 8
    rng = np.random.default_rng(4242)
    cuts = np.sort(rng.integers(0, nnz + 1, n_rows - 1))
    cuts[:10] = 0                                          # rows 0..9 empty
    rowptr = np.concatenate([[0], cuts, [nnz]]).astype(np.int64)
    gen = torch.Generator(device="cuda").manual_seed(4243)
    say(f"max nnz: {nnz} nonzeros, {n_rows} x {n_cols}")
    rp = torch.from_numpy(rowptr.astype(np.int32)).cuda()
    cl = torch.randint(0, n_cols, (nnz,), dtype=torch.int32, device="cuda", generator=gen)
    vl = torch.rand(nnz, dtype=torch.float32, device="cuda", generator=gen)
    xd = torch.randn(n_cols, F, dtype=torch.float32, device="cuda", generator=gen)
    xh = xd.cpu().numpy()
    # SpMM on the first, last, empty and random rows
    rows = np.unique(np.concatenate([[0, 5, 10, 11, n_rows - 1], rng.choice(n_rows, 40, replace=False)]))
    sub_ptr = np.concatenate([[0], np.cumsum(rowptr[rows + 1] - rowptr[rows])]).astype(np.int32)
    sub_col = np.concatenate([cl[rowptr[r]:rowptr[r + 1]].cpu().numpy() for r in rows]).astype(np.int32)
    sub_val = np.concatenate([vl[rowptr[r]:rowptr[r + 1]].cpu().numpy() for r in rows]).astype(np.float32)
    plan = cg.Plan(rp, nnz, F)
    try:
        Y = cg.spmm(rp, cl, vl, xd, plan=plan)
        Yr, Ar = oracle.spmm(sub_ptr, sub_col, sub_val, xh)
        assert scaled_error(Y[torch.from_numpy(rows).cuda()], Yr, Ar) <= TOL_F32
    finally:
        plan.close()
    del Y
    # transpose
    colptr, row_t, val_t, perm = cg.csr_to_csc(rp, cl, vl, n_cols)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    counts = torch.zeros(n_cols, dtype=torch.int64, device="cuda")
    for ch in cl.split(1 << 27):
        counts += torch.bincount(ch.long(), minlength=n_cols)
    ref_ptr = torch.zeros(n_cols + 1, dtype=torch.int64, device="cuda")
    ref_ptr[1:] = torch.cumsum(counts, 0)
    assert torch.equal(colptr.long(), ref_ptr)
    rp64 = rp.long()
    last_col, last_edge = -1, -1
    for s0 in range(0, nnz, 1 << 27):
        s1 = min(s0 + (1 << 27), nnz)
        slots = torch.arange(s0, s1, dtype=torch.int64, device="cuda")
        cslot = torch.searchsorted(ref_ptr[1:], slots, right=True)
        pc = perm[s0:s1].long()
        assert int(pc.min()) >= 0 and int(pc.max()) < nnz
        assert torch.equal(cl[pc].long(), cslot)
        assert torch.equal(row_t[s0:s1].long(), torch.searchsorted(rp64[1:], pc, right=True))
        assert torch.equal(val_t[s0:s1].view(torch.int32), vl[pc].view(torch.int32))
        same = cslot[1:] == cslot[:-1]
        assert bool((pc[1:][same] > pc[:-1][same]).all())
        if int(cslot[0]) == last_col:
            assert int(pc[0]) > last_edge
        last_col, last_edge = int(cslot[-1]), int(pc[-1])
        del slots, cslot, pc, same
    say("max nnz: transpose verified on every slot")
    # SpMM^T on sampled columns: the oracle sums each column's edges in CSR order
    G = torch.randn(n_rows, F, dtype=torch.float32, device="cuda", generator=gen)
    gh = G.cpu().numpy()
    plan_t = cg.Plan(colptr, nnz, F)
    try:
        dX = cg.spmm_t(colptr, row_t, val_t, G, plan_t=plan_t)
        for j in (0, 1, n_cols // 2, n_cols - 1):
            edges = torch.nonzero(cl == j).flatten()
            r = torch.searchsorted(rp64[1:], edges, right=True).cpu().numpy().astype(np.int32)
            v = vl[edges].cpu().numpy()
            ptr1 = np.array([0, r.size], np.int32)
            yr, ar = oracle.spmm(ptr1, r, v, gh)
            assert scaled_error(dX[j:j + 1], yr, ar) <= TOL_F32, j
    finally:
        plan_t.close()
    del cl, vl, colptr, row_t, val_t, perm, G
    torch.cuda.empty_cache()
