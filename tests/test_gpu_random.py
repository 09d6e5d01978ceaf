"""Seeded random sweep: graphs, feature widths, dtypes, balancer plans and head
layouts drawn at random (a fixed seed per case, so every run checks the same
cases), each operator of the hot path, the backward, the GSpMM variants, the
dense layer and the codec compared with the oracle.  It covers the combinations the parametrized tests do not spell out:
tiny and empty matrices, rectangular shapes, duplicates with unsorted columns,
hub rows against small neighbour groups, odd widths with 16-bit formats."""
import numpy as np
import pytest

import oracle
from paper_2103_00959_amd import synth

from gpu_util import TOL_ALPHA, TOL_F32, dev, features, graph_to_dev, say, scaled_error, to_f64, tol_for

pytestmark = pytest.mark.gpu

N_CASES = 120
KINDS = ["f32", "bf16", "f16"]


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _case(seed):
    rng = np.random.default_rng(9000 + seed)
    n_rows, n_cols = int(rng.integers(1, 400)), int(rng.integers(1, 400))
    dup = bool(rng.random() < 0.4)
    g = synth.random_csr(n_rows, n_cols, rng, mean_deg=float(rng.choice([0.5, 3.0, 12.0, 40.0])),
                         dup=dup, unsorted=bool(rng.random() < 0.5),
                         empty_frac=float(rng.choice([0.0, 0.3])))
    if rng.random() < 0.4 and n_rows > 1:
        # one hub row, far longer than the small neighbour groups below
        deg = np.diff(g.rowptr).astype(np.int64)
        hub = int(rng.integers(0, n_rows))
        deg[hub] = int(rng.integers(100, 700))
        rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
        cols = []
        for i in range(n_rows):
            lo, hi = g.rowptr[i], g.rowptr[i + 1]
            cols.append(g.col[lo:hi] if i != hub else rng.integers(0, n_cols, deg[hub]).astype(np.int32))
        col = np.concatenate(cols).astype(np.int32)
        g = synth.Graph(rowptr, col, rng.standard_normal(col.size).astype(np.float32), n_rows, n_cols)
    plan = [None, ("auto", 0), ("row_split", 0), ("neighbor_group", int(rng.choice([1, 2, 3, 5, 8, 16, 64])))][
        int(rng.integers(0, 4))]
    return rng, g, plan


def _plan(cg, rp, nnz, spec, max_feat, max_heads=0):
    if spec is None:
        return None
    return cg.Plan(rp, nnz, max_feat=max_feat, max_heads=max_heads, mode=spec[0], group_size=spec[1])


def _close(*plans):
    for p in plans:
        if p is not None:
            p.close()


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_spmm_gspmm_transpose(cg, seed):
    import torch
    rng, g, spec = _case(seed)
    F = int(rng.choice([1, 2, 3, 7, 8, 16, 33, 64, 100, 128, 256, 300]))
    xk = KINDS[int(rng.integers(0, 3))]
    out_f32 = bool(rng.random() < 0.5)
    say(f"random {seed}: {g.n_rows}x{g.n_cols} nnz={g.nnz} F={F} {xk} plan={spec}")
    rp, cl, vl = graph_to_dev(g)
    xh, xc, xd = features((g.n_cols, F), 300 + seed, xk)
    out_dtype = torch.float32 if out_f32 else xd.dtype
    plan = _plan(cg, rp, g.nnz, spec, F)
    try:
        Y = cg.spmm(rp, cl, vl, xd, plan=plan, out_dtype=out_dtype)
        Yr, Ar = oracle.spmm(g.rowptr, g.col, g.val, xh, x_dtype=xc)
        assert scaled_error(Y, Yr, Ar) <= tol_for(xk, "f32" if out_f32 else xk), "spmm"
        Ym = cg.gspmm(rp, cl, vl, xd, "mean", plan=plan, out_dtype=out_dtype)
        Ymr, Amr, _ = oracle.gspmm(g.rowptr, g.col, g.val, xh, "mean", n_cols=g.n_cols, x_dtype=xc)
        assert scaled_error(Ym, Ymr, Amr) <= tol_for(xk, "f32" if out_f32 else xk), "mean"
    finally:
        _close(plan)
    # transpose, bit for bit, and SpMM^T on it
    colptr, row_t, val_t, perm = cg.csr_to_csc(rp, cl, vl, g.n_cols)
    c_ref, r_ref, v_ref, p_ref = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
    assert np.array_equal(colptr.cpu().numpy(), c_ref)
    assert np.array_equal(row_t.cpu().numpy(), r_ref)
    assert np.array_equal(perm.cpu().numpy(), p_ref)
    assert np.array_equal(val_t.cpu().numpy().view(np.uint32), v_ref.view(np.uint32))
    gh, gc, gd = features((g.n_rows, F), 400 + seed, xk)
    plan_t = _plan(cg, colptr, g.nnz, spec, F)
    try:
        dX = cg.spmm_t(colptr, row_t, val_t, gd, plan_t=plan_t, out_dtype=out_dtype)
        dXr, dAr = oracle.spmm_t(g.rowptr, g.col, g.val, gh, g.n_cols, g_dtype=gc)
        assert scaled_error(dX, dXr, dAr) <= tol_for(xk, "f32" if out_f32 else xk), "spmm_t"
    finally:
        _close(plan_t)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_gat_forward_backward(cg, seed):
    import torch
    rng, g, spec = _case(seed)
    H = int(rng.choice([1, 2, 3, 4, 8]))
    D = int(rng.choice([1, 2, 5, 8, 16, 32, 64]))
    xk = ["f32", "bf16"][int(rng.integers(0, 2))]
    say(f"random gat {seed}: {g.n_rows}x{g.n_cols} nnz={g.nnz} H={H} D={D} {xk} plan={spec}")
    rp, cl, _ = graph_to_dev(g)
    srng = np.random.default_rng(500 + seed)
    sd = srng.standard_normal((g.n_rows, H)).astype(np.float32)
    ss = srng.standard_normal((g.n_cols, H)).astype(np.float32)
    xh, xc, xd = features((g.n_cols, H, D), 600 + seed, xk)
    plan = _plan(cg, rp, g.nnz, spec, H * D, max_heads=H)
    try:
        Y, a = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xd, 0.2, plan=plan, out_dtype=torch.float32,
                                return_alpha=True)
        Yr, Ar = oracle.gat(g.rowptr, g.col, sd, ss, xh.reshape(g.n_cols, H * D), H, D, slope=0.2, x_dtype=xc)
        assert scaled_error(Y.reshape(g.n_rows, H * D), Yr, Ar) <= tol_for(xk, "f32"), "gat"
        a_ref = oracle.edge_softmax(g.rowptr, g.col, sd, ss, slope=0.2)
        if g.nnz:
            rel = np.abs(to_f64(a).reshape(a_ref.shape) - a_ref) / a_ref
            assert rel.max() <= TOL_ALPHA, "alpha"
        a_s = cg.sddmm_edge_softmax(rp, cl, dev(sd), dev(ss), 0.2, plan=plan)
        if g.nnz:
            rel = np.abs(to_f64(a_s).reshape(a_ref.shape) - a_ref) / a_ref
            assert rel.max() <= TOL_ALPHA, "softmax"
    finally:
        _close(plan)
    # backward with the forward's fp32 weights
    alpha = a_ref.astype(np.float32)
    gh, gc, gd = features((g.n_rows, H, D), 700 + seed, xk)
    colptr, row_t, _, perm = oracle.csr_to_csc(g.rowptr, g.col, None, g.n_cols)
    cp_d, rt_d, pm_d = dev(colptr), dev(row_t), dev(perm)
    ref = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, xh.reshape(g.n_cols, H * D),
                              gh.reshape(g.n_rows, H * D), H, D, slope=0.2, x_dtype=xc, dy_dtype=gc)
    plan = _plan(cg, rp, g.nnz, spec, H * D, max_heads=H)
    plan_t = _plan(cg, cp_d, g.nnz, spec, H * D, max_heads=H)
    try:
        out = cg.gat_backward(rp, cl, cp_d, rt_d, pm_d, dev(sd), dev(ss), dev(alpha), xd, gd, 0.2,
                              plan=plan, plan_t=plan_t, dx_dtype=torch.float32)
        for k in ("dalpha", "dscore", "ds_dst", "ds_src"):
            assert scaled_error(out[k], ref[k], ref[k + "_abs"]) <= TOL_F32, k
        assert scaled_error(out["dX"].reshape(ref["dX"].shape), ref["dX"], ref["dX_abs"]) <= TOL_F32, "dX"
    finally:
        _close(plan, plan_t)


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_gspmm_max_and_messages(cg, seed):
    """Max with edge ids bit for bit (values rounded once to the output format, the first
    edge attaining each maximum); add / sub messages with the fp32 tolerance."""
    import torch
    rng, g, spec = _case(seed)
    F = int(rng.choice([1, 3, 8, 24, 64, 130]))
    xk = KINDS[int(rng.integers(0, 3))]
    yk = "f32" if rng.random() < 0.5 else xk
    say(f"random max {seed}: {g.n_rows}x{g.n_cols} nnz={g.nnz} F={F} {xk}->{yk} plan={spec}")
    rp, cl, vl = graph_to_dev(g)
    xh, xc, xd = features((g.n_cols, F), 800 + seed, xk)
    out_dtype = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[yk]
    plan = _plan(cg, rp, g.nnz, spec, F)
    try:
        Y, arg = cg.gspmm(rp, cl, vl, xd, "max", plan=plan, out_dtype=out_dtype, return_arg=True)
        Yr, _, ar = oracle.gspmm(g.rowptr, g.col, g.val, xh, "max", n_cols=g.n_cols, x_dtype=xc)
        code = {"f32": oracle.F32, "bf16": oracle.BF16, "f16": oracle.F16}[yk]
        want = oracle.decode(oracle.round_to(Yr, code), code)
        assert np.array_equal(to_f64(Y).reshape(Yr.shape), want.reshape(Yr.shape)), "max"
        assert np.array_equal(arg.cpu().numpy().reshape(ar.shape), ar), "argmax"
        compute = ["add", "sub"][int(rng.integers(0, 2))]
        reduce = ["sum", "mean"][int(rng.integers(0, 2))]
        Ya = cg.gspmm(rp, cl, vl, xd, reduce, plan=plan, out_dtype=torch.float32, compute=compute)
        Yar, Aar, _ = oracle.gspmm(g.rowptr, g.col, g.val, xh, reduce, n_cols=g.n_cols, x_dtype=xc,
                                   compute=compute)
        assert scaled_error(Ya, Yar, Aar) <= TOL_F32, (reduce, compute)
    finally:
        _close(plan)


@pytest.mark.parametrize("seed", range(N_CASES // 3))
def test_random_linear_and_codec(cg, seed):
    """Dense layer (any row count, k, m, bias and activation) with the fp32 tolerance; codec
    codes, stats and decodes bit for bit for random shapes, groups and bit widths."""
    import torch
    rng = np.random.default_rng(9500 + seed)
    n, k, m = int(rng.integers(1, 700)), int(rng.integers(1, 700)), int(rng.integers(1, 300))
    dt = ["bf16", "f16"][int(rng.integers(0, 2))]
    act = ["none", "relu", "elu"][int(rng.integers(0, 3))]
    code = oracle.BF16 if dt == "bf16" else oracle.F16
    to_bits = synth.f32_to_bf16_bits if dt == "bf16" else synth.f32_to_f16_bits
    tdt = torch.bfloat16 if dt == "bf16" else torch.float16
    xb = to_bits(rng.standard_normal((n, k)).astype(np.float32))
    wb = to_bits((rng.standard_normal((m, k)) / np.sqrt(k)).astype(np.float32))
    b = rng.standard_normal(m).astype(np.float32)
    say(f"random linear {seed}: {n}x{k}x{m} {dt} {act}")
    Y = cg.linear(dev(xb.view(np.int16)).view(tdt), dev(wb.view(np.int16)).view(tdt), bias=dev(b), act=act,
                  out_dtype=torch.float32)
    Yr, Ar = oracle.linear(xb, wb, b, act, x_dtype=code, w_dtype=code)
    assert scaled_error(Y, Yr, Ar) <= TOL_F32, "linear"
    bits = int(rng.integers(1, 9))
    G = int(rng.choice([64, 128, 256, 512]))
    rows, F = int(rng.integers(1, 600)), int(rng.integers(1, 700))
    at = KINDS[int(rng.integers(0, 3))]
    xh, xc, xd = features((rows, F), 950 + seed, at)
    cseed = int(rng.integers(0, 2**63))
    say(f"random codec {seed}: {rows}x{F} G={G} bits={bits} {at}")
    codes, stats = cg.act_compress(xd, bits, G, cseed)
    c_ref, s_ref = oracle.act_compress(xh, bits, G, cseed, a_dtype=xc)
    assert np.array_equal(codes.cpu().numpy().view(np.uint64), c_ref)
    assert np.array_equal(stats.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    y = cg.act_decompress(codes, stats, rows, F, bits, G)
    y_ref = oracle.act_decompress(c_ref, s_ref, rows, F, bits, G)
    assert np.array_equal(y.cpu().numpy().view(np.uint32), y_ref.view(np.uint32))
