"""GPU parity of the dense layer, the per-head scores, the aggregation
epilogues and the 2-layer GCN / GAT inference models against the oracle."""
import numpy as np
import pytest

import oracle
from paper_2103_00959_amd import synth

from gpu_util import TOL_16, TOL_F32, dev, features, graph_to_dev, say, scaled_error, to_f64

pytestmark = pytest.mark.gpu

# A model output may differ from the oracle's by one unit in the last place of
# each stored bf16 intermediate (Z1, H1, Z2: three roundings, 2^-7 relative
# each at most), propagated through the error scale E of gcn_forward /
# gat_forward; fp32 accumulation adds far less.
TOL_MODEL = 3 * 2.0 ** -7 + 1e-3


@pytest.fixture(scope="module")
def cg():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2103_00959_amd as m
    m.lib()
    return m


def _bf16_dev(x):
    import torch
    bits = synth.f32_to_bf16_bits(np.asarray(x, np.float32))
    return bits, dev(bits.view(np.int16)).view(torch.bfloat16)


def _f16_dev(x):
    import torch
    bits = synth.f32_to_f16_bits(np.asarray(x, np.float32))
    return bits, dev(bits.view(np.int16)).view(torch.float16)


# k covers one to 62 full 16-k steps (fewer, as many and one more than the loads
# kept in flight), a partial last step, and widths with only 4-byte or 2-byte alignment
@pytest.mark.parametrize("n,k,m", [(1, 16, 32), (300, 602, 128), (129, 64, 41), (1000, 128, 512),
                                   (5, 7, 3), (257, 24, 200), (64, 1000, 16), (70, 32, 96),
                                   (70, 48, 64), (131, 66, 33), (5, 0, 3)])
@pytest.mark.parametrize("dt,yt,act", [("bf16", "f32", "none"), ("bf16", "bf16", "relu"),
                                       ("f16", "f32", "elu"), ("f16", "f16", "none")])
def test_linear(cg, n, k, m, dt, yt, act):
    import torch
    rng = np.random.default_rng(n * 7 + k + m)
    mk = _bf16_dev if dt == "bf16" else _f16_dev
    code = oracle.BF16 if dt == "bf16" else oracle.F16
    xb, xd = mk(rng.standard_normal((n, k)))
    wb, wd = mk(rng.standard_normal((m, k)) / np.sqrt(k))
    b = rng.standard_normal(m).astype(np.float32)
    y_dtype = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[yt]
    Y = cg.linear(xd, wd, bias=dev(b), act=act, out_dtype=y_dtype)
    Yr, Ar = oracle.linear(xb, wb, b, act, x_dtype=code, w_dtype=code)
    err = scaled_error(Y, Yr, Ar)
    say(f"linear {n}x{k}x{m} {dt}->{yt} {act}: {err:.3g}")
    assert err <= (TOL_F32 if yt == "f32" else TOL_16)
    # without bias
    Y0 = cg.linear(xd, wd, out_dtype=torch.float32)
    Y0r, A0r = oracle.linear(xb, wb, None, "none", x_dtype=code, w_dtype=code)
    assert scaled_error(Y0, Y0r, A0r) <= TOL_F32


# vector path (heads of whole 16-byte vectors, H * D / VEC lanes a power of two up to 64):
# (4, 32), (8, 8), (1, 64), (2, 256), (4, 4), (16, 8); per-node fallback: the others
@pytest.mark.parametrize("H,D,zt", [(4, 32, "bf16"), (1, 41, "bf16"), (3, 5, "f32"), (8, 128, "f16"),
                                    (8, 8, "f32"), (1, 64, "bf16"), (2, 256, "bf16"), (4, 4, "f32"),
                                    (16, 8, "f16")])
def test_head_scores(cg, H, D, zt):
    rng = np.random.default_rng(H * D)
    n = 777
    zh, zc, zd = features((n, H, D), 60 + D, zt)
    a_s, a_d = rng.standard_normal((H, D)).astype(np.float32), rng.standard_normal((H, D)).astype(np.float32)
    s_src, s_dst = cg.head_scores(zd, dev(a_s), dev(a_d))
    ss, sd, sa, da = oracle.head_scores(zh.reshape(n, H * D), a_s, a_d, H, D, z_dtype=zc)
    assert scaled_error(s_src, ss, sa) <= TOL_F32
    assert scaled_error(s_dst, sd, da) <= TOL_F32


def _graph(kind, seed=0):
    rng = np.random.default_rng(seed)
    if kind == "small":
        return synth.random_csr(300, 300, rng, mean_deg=6, empty_frac=0.1)
    if kind == "hubs":
        g = synth.random_csr(3000, 3000, rng, mean_deg=3, empty_frac=0.3)
        deg = np.diff(g.rowptr).astype(np.int64)
        deg[[5, 1234, 2999]] = [1800, 2000, 700]
        rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int32)
        col = np.concatenate([np.sort(rng.choice(3000, d, replace=False)) for d in deg]).astype(np.int32)
        val = (rng.random(col.size) / np.repeat(np.maximum(deg, 1), deg)).astype(np.float32)
        return synth.Graph(rowptr, col, val, 3000, 3000)
    if kind == "cfg1":
        return synth.config_graph(1)
    raise KeyError(kind)


@pytest.mark.parametrize("kind", ["small", "hubs"])
@pytest.mark.parametrize("spec", [None, ("auto", 0), ("neighbor_group", 7)])
def test_aggregation_epilogues(cg, kind, spec):
    """act(aggregate + bias) for GSpMM sum / mean / max and the GAT aggregation."""
    import torch
    g = _graph(kind)
    rp, cl, vl = graph_to_dev(g)
    rng = np.random.default_rng(9)
    F = 64
    xh, xc, xd = features((g.n_cols, F), 71, "f32")
    b = rng.standard_normal(F).astype(np.float32)
    plan = None if spec is None else cg.Plan(rp, g.nnz, F, max_heads=4, mode=spec[0], group_size=spec[1])
    try:
        for red in ("sum", "mean", "max"):
            for act in ("relu", "elu", "none"):
                Y = cg.gspmm(rp, cl, vl, xd, red, plan=plan, bias=dev(b), act=act)
                Yr, Ar, _ = oracle.gspmm(g.rowptr, g.col, g.val, xh, red, n_cols=g.n_cols)
                Yr = oracle.epilogue(Yr, b, act)
                if red == "max":
                    # the maximum is exact; the epilogue adds one fp32 rounding
                    Ar = np.abs(Yr) + np.abs(b)[None, :]
                assert scaled_error(Y, Yr, Ar + np.abs(b)[None, :]) <= TOL_F32, (red, act)
        H, D = 4, 16
        sd = rng.standard_normal((g.n_rows, H)).astype(np.float32)
        ss = rng.standard_normal((g.n_cols, H)).astype(np.float32)
        xgh, xgc, xgd = features((g.n_cols, H, D), 72, "bf16")
        bg = rng.standard_normal(H * D).astype(np.float32)
        Yg = cg.gat_aggregate(rp, cl, dev(sd), dev(ss), xgd, 0.2, plan=plan, bias=dev(bg), act="elu",
                              out_dtype=torch.float32)
        Ygr, Agr = oracle.gat(g.rowptr, g.col, sd, ss, xgh.reshape(g.n_cols, H * D), H, D, slope=0.2,
                              x_dtype=xgc)
        Ygr = oracle.epilogue(Ygr, bg, "elu")
        assert scaled_error(Yg.reshape(g.n_rows, H * D), Ygr, Agr + np.abs(bg)[None, :]) <= TOL_F32
    finally:
        if plan is not None:
            plan.close()


def _gcn_params(rng, k, hid, out):
    W1b, W1 = _bf16_dev(rng.standard_normal((hid, k)) / np.sqrt(k))
    W2b, W2 = _bf16_dev(rng.standard_normal((out, hid)) / np.sqrt(hid))
    b1 = rng.standard_normal(hid).astype(np.float32) * 0.1
    b2 = rng.standard_normal(out).astype(np.float32) * 0.1
    host = dict(W1=W1b, b1=b1, W2=W2b, b2=b2)
    devp = dict(W1=W1, b1=dev(b1), W2=W2, b2=dev(b2))
    return host, devp


def _gat_params(rng, k, H, D, C):
    host, devp = {}, {}
    for name, shape, scale in (("W1", (H * D, k), 1 / np.sqrt(k)), ("W2", (C, H * D), 1 / np.sqrt(H * D))):
        host[name], devp[name] = _bf16_dev(rng.standard_normal(shape) * scale)
    for name, shape in (("a_src1", (H, D)), ("a_dst1", (H, D)), ("a_src2", (1, C)), ("a_dst2", (1, C))):
        host[name] = (rng.standard_normal(shape) / np.sqrt(shape[1])).astype(np.float32)
        devp[name] = dev(host[name])
    for name, size in (("b1", H * D), ("b2", C)):
        host[name] = (rng.standard_normal(size) * 0.1).astype(np.float32)
        devp[name] = dev(host[name])
    return host, devp


@pytest.mark.parametrize("kind", ["small", "hubs", "cfg1"])
@pytest.mark.parametrize("spec", [None, ("auto", 0), ("neighbor_group", 9)])
def test_gcn_model(cg, kind, spec):
    g = _graph(kind)
    rp, cl, vl = graph_to_dev(g)
    rng = np.random.default_rng(11)
    k, hid, out = 50, 32, 7
    xb, xd = _bf16_dev(rng.standard_normal((g.n_cols, k)))
    hp, dp = _gcn_params(rng, k, hid, out)
    plan = None if spec is None else cg.Plan(rp, g.nnz, max(k, hid, out), mode=spec[0], group_size=spec[1])
    try:
        Y = cg.gcn_forward(rp, cl, vl, xd, dp, plan=plan)
    finally:
        if plan is not None:
            plan.close()
    Yr, E = oracle.gcn_forward(g.rowptr, g.col, g.val, xb, hp)
    err = scaled_error(Y, Yr, E)
    say(f"gcn {kind} {spec}: {err:.3g}")
    assert err <= TOL_MODEL


@pytest.mark.parametrize("kind", ["small", "hubs", "cfg1"])
@pytest.mark.parametrize("spec", [None, ("auto", 0), ("neighbor_group", 9)])
def test_gat_model(cg, kind, spec):
    g = _graph(kind)
    rp, cl, _ = graph_to_dev(g)
    rng = np.random.default_rng(12)
    k, H, D, C = 40, 4, 8, 5
    xb, xd = _bf16_dev(rng.standard_normal((g.n_cols, k)))
    hp, dp = _gat_params(rng, k, H, D, C)
    plan = None if spec is None else cg.Plan(rp, g.nnz, max(k, H * D, C), max_heads=H, mode=spec[0],
                                            group_size=spec[1])
    try:
        Y = cg.gat_forward(rp, cl, xd, dp, 0.2, plan=plan)
    finally:
        if plan is not None:
            plan.close()
    Yr, E = oracle.gat_forward(g.rowptr, g.col, xb, hp, slope=0.2)
    err = scaled_error(Y, Yr, E)
    say(f"gat {kind} {spec}: {err:.3g}")
    assert err <= TOL_MODEL


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("n,F,G,at", [(50, 64, 64, "f32"), (300, 256, 256, "bf16"), (97, 300, 128, "bf16"),
                                      (33, 41, 64, "f16"), (1000, 128, 64, "f32"), (21, 2048, 1024, "bf16"),
                                      (7, 4096, 4096, "f32"), (13, 1024, 512, "f16"), (9, 2048, 2048, "bf16")])
def test_act_codec_bit_exact(cg, bits, n, F, G, at):
    """Codes, stats and decoded values equal the oracle's bit for bit (the same
    Philox stream, the same fp32 operations)."""
    import torch
    xh, xc, xd = features((n, F), 90 + F + bits, at)
    seed = 0x1234_5678_9ABC_DEF0 + bits
    codes, stats = cg.act_compress(xd, bits, G, seed)
    c_ref, s_ref = oracle.act_compress(xh, bits, G, seed, a_dtype=xc)
    assert np.array_equal(codes.cpu().numpy().view(np.uint64), c_ref)
    assert np.array_equal(stats.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    y = cg.act_decompress(codes, stats, n, F, bits, G)
    y_ref = oracle.act_decompress(c_ref, s_ref, n, F, bits, G)
    assert np.array_equal(y.cpu().numpy().view(np.uint32), y_ref.view(np.uint32))
    yb = cg.act_decompress(codes, stats, n, F, bits, G, out_dtype=torch.bfloat16)
    assert np.array_equal(yb.cpu().view(torch.int16).numpy().view(np.uint16),
                          oracle.round_to(y_ref.astype(np.float64), oracle.BF16))


@pytest.mark.parametrize("case", ["flat_index_whole", "flat_index_ragged", "clamp_whole", "clamp_ragged"])
def test_act_codec_constructed_cases(cg, case):
    """The hand-constructed codec inputs (each code on a threshold of its own uniform; the clamp
    where 255 + u rounds to 256) give the expected codes on both kernel paths (rows of whole
    16-byte aligned groups, ragged rows), bit for bit equal to the oracle's."""
    from codec_cases import clamp_case, flat_index_case
    if case.startswith("flat"):
        seed, bits = 0x5EED0001F00D, 1
        x, want = flat_index_case(seed, 3, 256 if case.endswith("whole") else 200)
    else:
        seed, bits = 11, 8
        x, _, want = clamp_case(seed, 0 if case.endswith("whole") else 8)
    n, F = x.shape
    codes, stats = cg.act_compress(dev(x), bits, 64, seed)
    c_ref, s_ref = oracle.act_compress(x, bits, 64, seed)
    assert np.array_equal(codes.cpu().numpy().view(np.uint64), c_ref)
    assert np.array_equal(stats.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    y = cg.act_decompress(codes, stats, n, F, bits, 64)
    assert np.array_equal(y.cpu().numpy(), want)


def test_act_codec_round_trip_on_aggregated_activations(cg):
    """Compress the GCN layer-1 activations of a graph at 2, 3, 4 bits: decoded
    values within one step of the originals, memory ratio as designed."""
    import torch
    g = _graph("hubs")
    rp, cl, vl = graph_to_dev(g)
    _, _, xd = features((g.n_cols, 256), 93, "f32")
    A = cg.spmm(rp, cl, vl, xd)
    for bits in (2, 3, 4):
        codes, stats = cg.act_compress(A, bits, 256, seed=5)
        y = cg.act_decompress(codes, stats, g.n_rows, 256, bits, 256)
        step = stats.view(-1, 2)[:, 1:2]
        assert bool(torch.all((y - A).abs() <= step * (1 + 1e-5) + 1e-7))
        ratio = A.numel() * 4 / (codes.numel() * 8 + stats.numel() * 4)
        assert abs(ratio - 32 / (bits + 64 / 256)) < 1e-6
