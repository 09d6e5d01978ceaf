"""The allocation-free transpose (cogdl_csr_to_csc_noalloc) against the transpose with a caller
workspace (cogdl_csr_to_csc), both called through the C ABI: every output bit for bit, on two
calls in a row on the same GPU (the second on a smaller graph, so it runs on what the first
left in the shared scratch), then without values and edge ids, then an empty graph."""
import ctypes

import numpy as np
import pytest

from paper_2103_00959_amd import synth

from gpu_util import dev, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _outs(torch, n_cols, nnz, with_val, with_perm):
    e = lambda n, dt: torch.full((n,), -7, dtype=dt, device="cuda")   # noqa: E731
    return (e(n_cols + 1, torch.int32), e(nnz, torch.int32),
            e(nnz, torch.float32) if with_val else None, e(nnz, torch.int32) if with_perm else None)


def _both(cg, g, with_val=True, with_perm=True):
    import torch
    L = cg.lib()
    rp, cl = dev(g.rowptr), dev(g.col)
    vl = dev(g.val) if with_val else None
    ref = _outs(torch, g.n_cols, g.nnz, with_val, with_perm)
    new = _outs(torch, g.n_cols, g.nnz, with_val, with_perm)
    ws_bytes = ctypes.c_size_t()
    assert L.cogdl_csr_to_csc_workspace(g.n_rows, g.n_cols, g.nnz, ctypes.byref(ws_bytes)) == 0
    ws = torch.empty(max(ws_bytes.value, 256), dtype=torch.uint8, device="cuda")
    P = cg._ptr
    s = cg._stream()
    say(f"noalloc transpose: n_rows {g.n_rows}, n_cols {g.n_cols}, nnz {g.nnz}, "
        f"values {with_val}, edge ids {with_perm}, workspace {ws_bytes.value} bytes")
    st = L.cogdl_csr_to_csc(g.n_rows, g.n_cols, g.nnz, P(rp), P(cl), P(vl), P(ref[0]), P(ref[1]),
                            P(ref[2]), P(ref[3]), P(ws), ws.numel(), s)
    assert st == 0
    st = L.cogdl_csr_to_csc_noalloc(g.n_rows, g.n_cols, g.nnz, P(rp), P(cl), P(vl), P(new[0]),
                                    P(new[1]), P(new[2]), P(new[3]), s)
    assert st == 0
    torch.cuda.synchronize()
    for a, b, name in zip(ref, new, ("colptr", "row_t", "val_t", "perm")):
        if a is None:
            continue
        assert torch.equal(a.view(torch.int32), b.view(torch.int32)), name
    # and the reference itself is the transpose (colptr = column counts, rows in CSR order)
    colptr = ref[0].cpu().numpy()
    assert np.array_equal(np.diff(colptr), np.bincount(g.col, minlength=g.n_cols))
    return ws_bytes.value


def test_noalloc_matches_workspace_transpose_twice(cg):
    rng = np.random.default_rng(2024)
    big = synth.random_csr(60000, 45000, rng, mean_deg=26, empty_frac=0.05, dup=True, unsorted=True)
    assert big.nnz > 1_400_000
    used = _both(cg, big)
    assert used <= 64 << 20
    small = synth.random_csr(3000, 2500, rng, mean_deg=5, empty_frac=0.1)
    assert small.nnz < big.nnz // 50
    _both(cg, small)
    _both(cg, small, with_val=False, with_perm=False)
    _both(cg, synth.config_graph(1))


def test_noalloc_empty_and_too_large(cg):
    import torch
    L = cg.lib()
    g = synth.Graph(np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), 5, 4)
    colptr = torch.full((5,), -1, dtype=torch.int32, device="cuda")
    z = dev(np.zeros(1, np.int32))
    assert L.cogdl_csr_to_csc_noalloc(5, 4, 0, cg._ptr(dev(g.rowptr)), cg._ptr(z), None,
                                      cg._ptr(colptr), cg._ptr(z), None, None, cg._stream()) == 0
    torch.cuda.synchronize()
    assert colptr.cpu().tolist() == [0] * 5
    # a graph past the scratch is refused before anything is launched, by the C ABI and the binding
    n = 2_000_000
    rp, cl = torch.arange(n + 1, dtype=torch.int32, device="cuda"), torch.zeros(n, dtype=torch.int32, device="cuda")
    out = torch.empty(n, dtype=torch.int32, device="cuda")
    assert L.cogdl_csr_to_csc_noalloc(n, 8, n, cg._ptr(rp), cg._ptr(cl), None, cg._ptr(colptr),
                                      cg._ptr(out), None, None, cg._stream()) == 6   # TOO_LARGE
    with pytest.raises(cg.CogdlError, match="static scratch holds"):
        cg.csr_to_csc_noalloc(rp, cl, None, 8)
