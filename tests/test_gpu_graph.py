"""The hot path under HIP graph capture: one step (plan rebuild, SpMM, CSR -> CSC,
plan rebuild on the CSC, SpMM^T, fused GAT aggregation with alpha) captured once
and replayed several times, with unrelated eager work on the same buffers'
neighbours in between; every replay must equal the eager step bit for bit (the
library launches only kernels in these calls: no memset or copy nodes, and its
results are deterministic)."""
import numpy as np
import pytest

from paper_2103_00959_amd import synth

from gpu_util import dev, features, graph_to_dev, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _graph(seed):
    rng = np.random.default_rng(seed)
    g = synth.random_csr(2000, 2000, rng, mean_deg=6, empty_frac=0.1)
    deg = np.diff(g.rowptr).astype(np.int64)
    deg[[3, 1500]] = [900, 1300]                       # split rows under group size 64
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
    col = np.concatenate([np.sort(rng.choice(2000, d, replace=False)) for d in deg]).astype(np.int32)
    return synth.Graph(rowptr, col, rng.standard_normal(col.size).astype(np.float32), 2000, 2000)


@pytest.mark.parametrize("seed,sliced", [(1, False), (2, False), (3, True), (4, True)])
def test_step_under_graph_capture(cg, seed, sliced):
    import torch
    g = _graph(seed)
    N, E = g.n_rows, g.nnz
    F, H, D = 256, 4, 64
    rp, cl, vl = graph_to_dev(g)
    _, _, X = features((N, F), 10 + seed, "bf16")
    _, _, G = features((N, F), 20 + seed, "bf16")
    _, _, Xg = features((N, H, D), 30 + seed, "bf16")
    rng = np.random.default_rng(40 + seed)
    sd = dev(rng.standard_normal((N, H)).astype(np.float32))
    ss = dev(rng.standard_normal((N, H)).astype(np.float32))
    Y = torch.empty((N, F), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty_like(Y)
    Yg = torch.empty((N, H, D), dtype=torch.bfloat16, device="cuda")
    alpha = torch.empty((E, H), dtype=torch.float32, device="cuda")
    colptr = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    row_t = torch.empty(E, dtype=torch.int32, device="cuda")
    val_t = torch.empty(E, dtype=torch.float32, device="cuda")
    perm = torch.empty(E, dtype=torch.int32, device="cuda")
    ws = torch.empty(cg.csr_to_csc_workspace(N, N, E), dtype=torch.uint8, device="cuda")
    L = cg.lib()
    plan = cg.Plan(rp, E, max_feat=F, max_heads=H, mode="neighbor_group", group_size=64,
                   **(dict(col=cl, n_cols=N, slice_min=32) if sliced else {}))

    def csc():
        cg._check(L.cogdl_csr_to_csc(N, N, E, cg._ptr(rp), cg._ptr(cl), cg._ptr(vl), cg._ptr(colptr),
                                     cg._ptr(row_t), cg._ptr(val_t), cg._ptr(perm), cg._ptr(ws),
                                     ws.numel(), cg._stream()), "csr_to_csc")

    csc()
    plan_t = cg.Plan(colptr, E, max_feat=F, max_heads=H, mode="neighbor_group", group_size=64,
                     **(dict(col=row_t, n_cols=N, slice_min=32) if sliced else {}))

    def step():
        plan.rebuild(rp)
        cg.spmm(rp, cl, vl, X, plan=plan, out=Y)
        csc()
        plan_t.rebuild(colptr)
        cg.spmm_t(colptr, row_t, val_t, G, plan_t=plan_t, out=dX)
        cg.gat_aggregate(rp, cl, sd, ss, Xg, 0.2, plan=plan, out=Yg, alpha_out=alpha)

    outs = (Y, dX, Yg, alpha, colptr, row_t, val_t, perm)
    try:
        step()
        torch.cuda.synchronize()
        ref = [t.clone() for t in outs]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()                                   # warm on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        for rep in range(3):
            for t in outs:
                t.zero_()                            # the replay must rewrite every output
            Y2 = cg.spmm(rp, cl, vl, G, plan=plan)   # eager work between the replays
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            say(f"graph replay {rep}")
            for a, b in zip(outs, ref):
                assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                                   b.view(torch.int16) if b.dtype == torch.bfloat16 else b), rep
            del Y2
        del graph
    finally:
        plan.close()
        plan_t.close()
