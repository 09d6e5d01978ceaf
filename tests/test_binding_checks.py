"""Size checks of the Python binding (no GPU needed).

The C ABI takes bare device pointers, so it cannot see how large a tensor is;
the binding checks every size the library would read or write through before
it checks devices or launches anything.  These tests pass host tensors of the
wrong size and expect a CogdlError that names the size problem; a tensor of
the right size would get as far as the device check ("must be a CUDA
tensor"), which is how each test knows the size check fired first.  No kernel
is launched (there is no GPU here)."""
import pytest
import torch

import paper_2103_00959_amd as cg

i32, f32, bf16 = torch.int32, torch.float32, torch.bfloat16


def graph(n_rows=4, nnz=6):
    rowptr = torch.tensor([0, 2, 3, 5, 6][: n_rows + 1], dtype=i32)
    col = torch.zeros(nnz, dtype=i32)
    return rowptr, col


def raises_size(fn, pattern):
    with pytest.raises(cg.CogdlError, match=pattern):
        fn()


def reaches_device_check(fn):
    with pytest.raises(cg.CogdlError, match="CUDA"):
        fn()


def test_spmm_sizes():
    rp, col = graph()
    X = torch.zeros(5, 8, dtype=f32)
    reaches_device_check(lambda: cg.spmm(rp, col, torch.zeros(6), X))
    raises_size(lambda: cg.spmm(rp, col, torch.zeros(5), X), "val has 5 elements, expected 6")
    raises_size(lambda: cg.spmm(rp, col, None, X, out=torch.zeros(4, 7)), "out has 28 elements, expected 32")
    raises_size(lambda: cg.spmm(rp, col, None, torch.zeros(5, 8, 2)), "X must be")
    raises_size(lambda: cg.spmm(rp.view(1, -1), col, None, X), "rowptr must have 1 dimensions")
    raises_size(lambda: cg.spmm(torch.zeros(0, dtype=i32), col, None, X), "at least one entry")
    raises_size(lambda: cg.spmm(rp, col.view(2, 3), None, X), "col must have 1 dimensions")
    raises_size(lambda: cg.spmm(rp, col, None, X.numpy()), "must be a torch tensor")


def test_gspmm_sizes():
    rp, col = graph()
    X = torch.zeros(5, 8, dtype=f32)
    reaches_device_check(lambda: cg.gspmm(rp, col, None, X, "max", return_arg=True))
    raises_size(lambda: cg.gspmm(rp, col, None, X, "max", arg=torch.zeros(4, 4, dtype=i32)),
                "arg has 16 elements, expected 32")
    raises_size(lambda: cg.gspmm(rp, col, None, X, bias=torch.zeros(7)), "bias has 7 elements, expected 8")
    raises_size(lambda: cg.gspmm(rp, col, torch.zeros(7), X), "val has 7 elements")
    raises_size(lambda: cg.gspmm(rp, col, None, X, out=torch.zeros(3, 8)), "out has 24 elements")
    with pytest.raises(ValueError):
        cg.gspmm(rp, col, None, X, "sum", arg=torch.zeros(4, 8, dtype=i32))


def test_transpose_and_spmm_t_sizes():
    rp, col = graph()
    reaches_device_check(lambda: cg.csr_to_csc(rp, col, torch.zeros(6), 5))
    raises_size(lambda: cg.csr_to_csc(rp, col, torch.zeros(4), 5), "val has 4 elements, expected 6")
    raises_size(lambda: cg.csr_to_csc(rp, col, None, -1), "n_cols must be >= 0")
    colptr, row_t = torch.zeros(6, dtype=i32), torch.zeros(6, dtype=i32)
    G = torch.zeros(4, 8, dtype=f32)
    reaches_device_check(lambda: cg.spmm_t(colptr, row_t, torch.zeros(6), G))
    raises_size(lambda: cg.spmm_t(colptr, row_t, torch.zeros(5), G), "val_t has 5 elements")
    raises_size(lambda: cg.spmm_t(colptr, row_t, None, G, out=torch.zeros(4, 8)), "out has 32 elements, expected 40")


def test_softmax_and_gat_sizes():
    rp, col = graph()
    sd, ss = torch.zeros(4, 2), torch.zeros(5, 2)
    X = torch.zeros(5, 2, 3, dtype=f32)
    reaches_device_check(lambda: cg.sddmm_edge_softmax(rp, col, sd, ss))
    raises_size(lambda: cg.sddmm_edge_softmax(rp, col, torch.zeros(3, 2), ss), r"s_dst must be \[4, 2\]")
    raises_size(lambda: cg.sddmm_edge_softmax(rp, col, torch.zeros(4, 3), ss), r"s_dst must be \[4, 2\]")
    raises_size(lambda: cg.sddmm_edge_softmax(rp, col, sd, ss, out=torch.zeros(6, 3)), "alpha has 18 elements")
    reaches_device_check(lambda: cg.gat_aggregate(rp, col, sd, ss, X))
    raises_size(lambda: cg.gat_aggregate(rp, col, sd, torch.zeros(4, 2), X), r"s_src must be \[5, 2\]")
    raises_size(lambda: cg.gat_aggregate(rp, col, sd, ss, X.view(5, 6)), "X must have 3 dimensions")
    raises_size(lambda: cg.gat_aggregate(rp, col, sd, ss, X, out=torch.zeros(4, 2, 2)), "out has 16 elements")
    raises_size(lambda: cg.gat_aggregate(rp, col, sd, ss, X, alpha_out=torch.zeros(6, 1)),
                "alpha_out has 6 elements, expected 12")
    raises_size(lambda: cg.gat_aggregate(rp, col, sd, ss, X, bias=torch.zeros(5)), "bias has 5 elements")
    raises_size(lambda: cg.gat_aggregate(rp, col, None, None, X, alpha_in=torch.zeros(6, 1)),
                "alpha_in has 6 elements, expected 12")
    reaches_device_check(lambda: cg.gat_aggregate(rp, col, None, None, X, alpha_in=torch.zeros(6, 2)))


def test_sddmm_dot_and_backward_sizes():
    rp, col = graph()
    P, Q = torch.zeros(4, 2, 3), torch.zeros(5, 2, 3)
    reaches_device_check(lambda: cg.sddmm_dot(rp, col, P, Q))
    raises_size(lambda: cg.sddmm_dot(rp, col, torch.zeros(3, 2, 3), Q), "P has 3 rows")
    raises_size(lambda: cg.sddmm_dot(rp, col, P, torch.zeros(5, 2, 4)), "same H and D")
    raises_size(lambda: cg.sddmm_dot(rp, col, P, Q, out=torch.zeros(6)), "out has 6 elements, expected 12")
    X, dY = torch.zeros(5, 2, 3), torch.zeros(4, 2, 3)
    colptr, row_t, perm = torch.zeros(6, dtype=i32), torch.zeros(6, dtype=i32), torch.zeros(6, dtype=i32)
    sd, ss, al = torch.zeros(4, 2), torch.zeros(5, 2), torch.zeros(6, 2)
    args = dict(rowptr=rp, col=col, colptr=colptr, row_t=row_t, perm=perm, s_dst=sd, s_src=ss, alpha=al,
                X=X, dY=dY)
    reaches_device_check(lambda: cg.gat_backward(**args))
    for key, bad, pat in (("colptr", torch.zeros(5, dtype=i32), "colptr has 5 elements"),
                          ("row_t", torch.zeros(5, dtype=i32), "row_t has 5 elements"),
                          ("perm", torch.zeros(7, dtype=i32), "perm has 7 elements"),
                          ("alpha", torch.zeros(6, 1), "alpha has 6 elements"),
                          ("s_src", torch.zeros(4, 2), r"s_src must be \[5, 2\]"),
                          ("dY", torch.zeros(3, 2, 3), r"dY must be \[4, 2, 3\]")):
        raises_size(lambda: cg.gat_backward(**dict(args, **{key: bad})), pat)
    raises_size(lambda: cg.gat_backward(**args, out={"dX": torch.zeros(5, 2, 2)}), "dX has 20 elements")
    raises_size(lambda: cg.gat_backward(**args, out={"ds_src": torch.zeros(4, 2)}), "ds_src has 8 elements")
    raises_size(lambda: cg.gat_backward(**args, out={"grad": torch.zeros(1)}), "unknown output")
    # the per-edge outputs may be left out, no other
    reaches_device_check(lambda: cg.gat_backward(**args, out={"dalpha": None, "dscore": None}))
    raises_size(lambda: cg.gat_backward(**args, out={"ds_dst": None}), "output 'ds_dst' is required")
    # the weights rebuilt from row softmax states instead of alpha
    st = torch.zeros(4, 2, 2)
    reaches_device_check(lambda: cg.gat_backward(**dict(args, alpha=None), row_stats=st))
    raises_size(lambda: cg.gat_backward(**dict(args, alpha=None), row_stats=torch.zeros(4, 2, 1)),
                "row_stats has 8 elements, expected 16")
    raises_size(lambda: cg.gat_backward(**args, row_stats=st), "exactly one of alpha and row_stats")
    raises_size(lambda: cg.gat_backward(**dict(args, alpha=None)), "exactly one of alpha and row_stats")


def test_gat_stats_forward_sizes():
    rp, col = graph()
    sd, ss = torch.zeros(4, 2), torch.zeros(5, 2)
    X = torch.zeros(5, 2, 8, dtype=f32)
    reaches_device_check(lambda: cg.gat_aggregate_stats(rp, col, sd, X, s_src=ss))
    reaches_device_check(lambda: cg.gat_aggregate_stats(rp, col, sd, X, a_src=torch.zeros(2, 8)))
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X), "exactly one of s_src and a_src")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X, s_src=ss, a_src=torch.zeros(2, 8)),
                "exactly one of s_src and a_src")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X, a_src=torch.zeros(2, 7)),
                "a_src has 14 elements, expected 16")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X, s_src=torch.zeros(4, 2)), r"s_src must be \[5, 2\]")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, torch.zeros(4, 3), X, s_src=ss), r"s_dst must be \[4, 2\]")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X, s_src=ss, stats_out=torch.zeros(4, 2)),
                "stats_out has 8 elements, expected 16")
    raises_size(lambda: cg.gat_aggregate_stats(rp, col, sd, X, s_src=ss, out=torch.zeros(4, 2, 7)),
                "out has 56 elements, expected 64")


def test_dense_and_codec_sizes():
    X, W = torch.zeros(6, 16, dtype=bf16), torch.zeros(3, 16, dtype=bf16)
    reaches_device_check(lambda: cg.linear(X, W))
    raises_size(lambda: cg.linear(X, W, bias=torch.zeros(4)), "bias has 4 elements, expected 3")
    raises_size(lambda: cg.linear(X, W, out=torch.zeros(6, 4)), "out has 24 elements, expected 18")
    raises_size(lambda: cg.linear(X, torch.zeros(3, 15, dtype=bf16)), "same dtype")
    Z = torch.zeros(6, 2, 8, dtype=bf16)
    reaches_device_check(lambda: cg.head_scores(Z, torch.zeros(2, 8), torch.zeros(2, 8)))
    raises_size(lambda: cg.head_scores(Z, torch.zeros(2, 7), torch.zeros(2, 8)), "a_src has 14 elements")
    A = torch.zeros(4, 128, dtype=f32)
    words, nst = cg.act_codec_size(4, 128, 2, 64)
    reaches_device_check(lambda: cg.act_compress(A, 2, 64, 1))
    raises_size(lambda: cg.act_compress(A, 2, 64, 1, codes=torch.zeros(words - 1, dtype=torch.int64)),
                f"codes has {words - 1} elements, needs at least {words}")
    raises_size(lambda: cg.act_compress(A, 2, 64, 1, stats=torch.zeros(nst - 1)), "stats has")
    codes, stats = torch.zeros(words, dtype=torch.int64), torch.zeros(nst)
    reaches_device_check(lambda: cg.act_decompress(codes, stats, 4, 128, 2, 64))
    raises_size(lambda: cg.act_decompress(codes[:-1], stats, 4, 128, 2, 64), "codes has")
    raises_size(lambda: cg.act_decompress(codes, stats, 4, 128, 2, 64, out=torch.zeros(4, 127)),
                "out has 508 elements")


def test_plan_sizes():
    rp, col = graph()
    reaches_device_check(lambda: cg.Plan(rp, 6, max_feat=8))
    raises_size(lambda: cg.Plan(rp, 6, max_feat=8, col=torch.zeros(5, dtype=i32), n_cols=5),
                "col has 5 elements, expected 6")
    raises_size(lambda: cg.Plan(rp, 6, max_feat=8, col=col), "needs n_cols")
    raises_size(lambda: cg.Plan(rp, 6, max_feat=8, mode="fastest"), "mode must be one of")

    class FakePlan:   # a plan object as the binding sees it, without a device
        n_rows, nnz = 4, 6
    p = cg.Plan.__new__(cg.Plan)
    p.n_rows, p.nnz, p.sliced, p._h = 4, 6, True, None
    raises_size(lambda: p.rebuild(torch.zeros(4, dtype=i32)), "rowptr has 4 elements, expected 5")
    raises_size(lambda: p.rebuild(rp, torch.zeros(7, dtype=i32)), "col has 7 elements, expected 6")
    other = FakePlan()
    other.n_rows = 3
    raises_size(lambda: cg.spmm(rp, col, None, torch.zeros(5, 8), plan=other), "plan was built for 3 rows")
    raises_size(lambda: cg.spmm_t(torch.zeros(6, dtype=i32), col, None, torch.zeros(4, 8), plan_t=FakePlan()),
                "plan_t was built for 4 rows")
