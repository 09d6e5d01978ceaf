"""Pins for the CPU oracle: each checks it against something other than itself
(hand-derived values, closed forms, invariants, dense/scipy special cases,
brute force on tiny graphs), chosen so that a dropped term, a wrong sign, a
wrong index or a transposed operand fails at least one of them."""
import json
from fractions import Fraction
import math
import os

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from paper_2103_00959_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _dense(g):
    A = np.zeros((g.n_rows, g.n_cols))
    rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
    vals = np.ones(g.col.size) if g.val is None else g.val.astype(np.float64)
    np.add.at(A, (rows, g.col), vals)          # duplicates add up
    return A


def _graphs(seed=0):
    rng = np.random.default_rng(seed)
    yield synth.random_csr(37, 37, rng, mean_deg=3)
    yield synth.random_csr(50, 23, rng, mean_deg=5, dup=True, unsorted=True, empty_frac=0.2)
    yield synth.random_csr(23, 61, rng, mean_deg=8, unsorted=True)
    yield synth.random_csr(200, 150, rng, mean_deg=12, dup=True, empty_frac=0.1)
    yield synth.random_csr(1, 5, rng, mean_deg=4)


# ------------------------------------------------------------ formats

def test_decode_known_patterns():
    bf = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x0000, 0x8000], dtype=np.uint16)
    exp_bf = [1.0, -2.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, 0.0, -0.0]
    assert oracle.decode(bf, oracle.BF16).tolist() == exp_bf
    hf = np.array([0x3C00, 0x0001, 0x7BFF, 0xC400, 0x0400, 0x3555], dtype=np.uint16)
    exp_hf = [1.0, 2.0 ** -24, 65504.0, -4.0, 2.0 ** -14, 1365.0 / 4096.0]
    assert oracle.decode(hf, oracle.F16).tolist() == exp_hf


def test_round_bf16_ties_and_no_double_rounding():
    one = 1.0
    cases = [
        (one + 2 ** -8, 0x3F80),                 # tie -> even (1.0)
        (one + 3 * 2 ** -8, 0x3F82),             # tie -> even (odd neighbour skipped)
        (one + 2 ** -8 + 2 ** -30, 0x3F81),      # just above the tie; float-first would give 0x3F80
        (-(one + 2 ** -7), 0xBF81),
        (2.0 ** -133, 0x0001),                   # smallest subnormal
        (2.0 ** -134, 0x0000),                   # tie between 0 and 2^-133 -> even
        (3.0e38 * 10, 0x7F80),                   # overflow -> inf
    ]
    got = oracle.round_to(np.array([c[0] for c in cases]), oracle.BF16)
    assert got.tolist() == [c[1] for c in cases]


def test_round_f16_matches_numpy_half():
    rng = np.random.default_rng(3)
    v = np.concatenate([rng.standard_normal(5000) * 10.0 ** rng.integers(-9, 5, 5000),
                        [65504.0, 65519.9, 65520.0, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -24]])
    got = oracle.round_to(v, oracle.F16)
    with np.errstate(over="ignore"):
        want = v.astype(np.float16).view(np.uint16)  # numpy rounds double -> half directly
    assert np.array_equal(got, want)


def test_round_f32_is_cast():
    v = np.random.default_rng(4).standard_normal(1000) * 1e3
    assert np.array_equal(oracle.round_to(v, oracle.F32), v.astype(np.float32))


# ------------------------------------------------------------ balancer

def test_balancer_modes_golden():
    with open(os.path.join(GOLDEN, "balancer_modes.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        d = np.array(c["degrees"], dtype=np.int64)
        rowptr = np.concatenate([[0], np.cumsum(d)]).astype(np.int32)
        assert oracle.balance_mode(rowptr, int(d.sum())) == c["mode"], c["name"]


@pytest.mark.parametrize("G", [1, 2, 3, 7, 64])
def test_neighbor_groups_tile_edges(G):
    for g in _graphs(1):
        for mode in (oracle.ROW_SPLIT, oracle.NEIGHBOR_GROUP):
            groups = oracle.neighbor_groups(g.rowptr, G, mode)
            d = np.diff(g.rowptr)
            if mode == oracle.ROW_SPLIT:
                assert len(groups) == g.n_rows
            else:
                assert len(groups) == int(np.sum(np.maximum(1, -(-d // G))))
                assert np.all(groups[:, 2] - groups[:, 1] <= G)
            assert np.all(np.diff(groups[:, 0]) >= 0) and np.all(np.diff(groups[:, 1]) >= 0)
            cover = np.zeros(g.nnz, dtype=np.int64)
            for r, b, e in groups:
                assert g.rowptr[r] <= b <= e <= g.rowptr[r + 1]
                cover[b:e] += 1
            assert np.all(cover == 1)


# ------------------------------------------------------------ SpMM

def test_spmm_golden_hand_example():
    with open(os.path.join(GOLDEN, "csr_dups_unsorted.json")) as f:
        c = json.load(f)
    X = np.array(c["X"], dtype=np.float32)
    Y, A = oracle.spmm(c["rowptr"], c["col"], np.array(c["val"], np.float32), X)
    assert Y.tolist() == c["Y"]


def test_spmm_dense_special_case():
    rng = np.random.default_rng(5)
    for g in _graphs(2):
        X = rng.standard_normal((g.n_cols, 7)).astype(np.float32)
        Y, Abs = oracle.spmm(g.rowptr, g.col, g.val, X)
        D = _dense(g)
        np.testing.assert_allclose(Y, D @ X.astype(np.float64), rtol=1e-12, atol=1e-12)
        Dabs = np.zeros_like(D)
        rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
        np.add.at(Dabs, (rows, g.col), np.abs(g.val.astype(np.float64)))
        np.testing.assert_allclose(Abs, Dabs @ np.abs(X.astype(np.float64)), rtol=1e-12)


def test_spmm_scipy_cross_check():
    rng = np.random.default_rng(6)
    g = synth.random_csr(2000, 1500, rng, mean_deg=9, dup=True, unsorted=True)
    X = rng.standard_normal((g.n_cols, 33)).astype(np.float32)
    Y, _ = oracle.spmm(g.rowptr, g.col, g.val, X)
    S = sp.csr_matrix((g.val.astype(np.float64), g.col, g.rowptr), shape=(g.n_rows, g.n_cols))
    np.testing.assert_allclose(Y, S @ X.astype(np.float64), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("n", [2, 3, 4])
def test_spmm_exhaustive_patterns(n):
    """Every directed pattern on n nodes (2^(n*n) graphs, self pairs included),
    batched as one block-diagonal graph, against dense products per block."""
    rng = np.random.default_rng(7 + n)
    n_pat = 1 << (n * n)
    bits = ((np.arange(n_pat)[:, None] >> np.arange(n * n)[None, :]) & 1).astype(bool)
    mats = bits.reshape(n_pat, n, n)
    W = rng.standard_normal((n_pat, n, n)) * mats
    W = W.astype(np.float32)
    rowptr = np.concatenate([[0], np.cumsum(mats.reshape(-1, n).sum(1))]).astype(np.int32)
    blk, r, c = np.nonzero(mats)
    col = (blk * n + c).astype(np.int32)
    val = W[blk, r, c]
    F = 3
    X = rng.standard_normal((n_pat * n, F)).astype(np.float32)
    Y, _ = oracle.spmm(rowptr, col, val, X)
    want = np.einsum("bij,bjf->bif", W.astype(np.float64), X.reshape(n_pat, n, F).astype(np.float64))
    np.testing.assert_allclose(Y.reshape(n_pat, n, F), want, rtol=1e-12, atol=1e-13)


def _regular_graphs():
    def from_adj(nbrs, n):
        keys = np.unique(np.array([i * n + j for i in range(n) for j in nbrs(i)] +
                                  [i * n + i for i in range(n)], dtype=np.int64))
        return synth._csr_from_keys(keys, n, n)
    yield 2, from_adj(lambda i: [(i + 1) % 11, (i - 1) % 11], 11)                   # cycle C11
    yield 6, from_adj(lambda i: [j for j in range(7) if j != i], 7)                  # K7
    yield 5, from_adj(lambda i: [i ^ (1 << b) for b in range(5)], 32)                # hypercube Q5
    yield 6, from_adj(lambda i: [(i + s) % 40 for s in (1, 3, 7, -1, -3, -7)], 40)  # circulant


def test_sym_norm_ones_invariant():
    """D^-1/2 (A+I) D^-1/2 applied to the ones vector on a k-regular graph is 1."""
    for k, g in _regular_graphs():
        assert np.all(np.diff(g.rowptr) == k + 1)
        g.val = synth.sym_norm_values(g)
        Y, _ = oracle.spmm(g.rowptr, g.col, g.val, np.ones((g.n_cols, 2), np.float32))
        # only the fp32 storage of 1/(k+1) is inexact
        assert np.max(np.abs(Y - 1.0)) <= (k + 1) * 2.0 ** -24


def test_row_norm_ones_invariant():
    rng = np.random.default_rng(8)
    g = synth.random_csr(300, 300, rng, mean_deg=6)
    keep = np.diff(g.rowptr) > 0
    g.val = synth.row_norm_values(g)
    Y, _ = oracle.spmm(g.rowptr, g.col, g.val, np.ones((g.n_cols, 1), np.float32))
    d = np.diff(g.rowptr)
    assert np.all(np.abs(Y[keep, 0] - 1.0) <= d[keep] * 2.0 ** -24)
    assert np.all(Y[~keep] == 0)


def test_spmm_identity_bit_exact_all_dtypes():
    rng = np.random.default_rng(9)
    n = 97
    rowptr = np.arange(n + 1, dtype=np.int32)
    col = np.arange(n, dtype=np.int32)
    val = np.ones(n, dtype=np.float32)
    x32 = rng.standard_normal((n, 9)).astype(np.float32)
    for dt, X in ((oracle.F32, x32), (oracle.BF16, synth.f32_to_bf16_bits(x32)),
                  (oracle.F16, synth.f32_to_f16_bits(x32))):
        Y, _ = oracle.spmm(rowptr, col, val, X, x_dtype=dt)
        assert np.array_equal(oracle.round_to(Y, dt), X)


def test_spmm_linearity():
    rng = np.random.default_rng(10)
    g = synth.random_csr(120, 90, rng, mean_deg=7, dup=True)
    # small integers keep a*X + b*Z exact in fp32, so only the operator is tested
    X = rng.integers(-8, 9, (90, 5)).astype(np.float32)
    Z = rng.integers(-8, 9, (90, 5)).astype(np.float32)
    a, b = np.float32(0.5), np.float32(-2.0)
    Yx, Ax = oracle.spmm(g.rowptr, g.col, g.val, X)
    Yz, Az = oracle.spmm(g.rowptr, g.col, g.val, Z)
    Yc, _ = oracle.spmm(g.rowptr, g.col, g.val, a * X + b * Z)
    scale = np.abs(a) * Ax + np.abs(b) * Az + 1e-300
    assert np.max(np.abs(Yc - (a * Yx + b * Yz)) / scale) < 1e-13


def test_spmm_16bit_inputs_decode_independently():
    rng = np.random.default_rng(11)
    g = synth.random_csr(64, 40, rng, mean_deg=5)
    x32 = rng.standard_normal((40, 8)).astype(np.float32)
    bf = synth.f32_to_bf16_bits(x32)
    via_numpy = (bf.astype(np.uint32) << 16).view(np.float32)
    Yb, _ = oracle.spmm(g.rowptr, g.col, g.val, bf, x_dtype=oracle.BF16)
    Yf, _ = oracle.spmm(g.rowptr, g.col, g.val, via_numpy)
    assert np.array_equal(Yb, Yf)
    hf = synth.f32_to_f16_bits(x32)
    Yh, _ = oracle.spmm(g.rowptr, g.col, g.val, hf, x_dtype=oracle.F16)
    Yf, _ = oracle.spmm(g.rowptr, g.col, g.val, hf.view(np.float16).astype(np.float32))
    assert np.array_equal(Yh, Yf)


def test_spmm_selected_rows_match_full():
    rng = np.random.default_rng(12)
    g = synth.random_csr(300, 200, rng, mean_deg=6, empty_frac=0.1)
    X = rng.standard_normal((200, 4)).astype(np.float32)
    Y, A = oracle.spmm(g.rowptr, g.col, g.val, X)
    sel = np.array([299, 0, 17, 17, 150], dtype=np.int32)
    Ys, As = oracle.spmm(g.rowptr, g.col, g.val, X, rows=sel)
    assert np.array_equal(Ys, Y[sel]) and np.array_equal(As, A[sel])


def test_spmm_empty_graph_and_zero_width():
    rowptr = np.zeros(6, dtype=np.int32)
    Y, _ = oracle.spmm(rowptr, np.zeros(0, np.int32), np.zeros(0, np.float32),
                       np.ones((4, 3), np.float32))
    assert Y.shape == (5, 3) and np.all(Y == 0)


# ------------------------------------------------------------ CSR -> CSC

def test_csc_golden_stable_with_duplicates():
    with open(os.path.join(GOLDEN, "csr_dups_unsorted.json")) as f:
        c = json.load(f)
    colptr, row_t, val_t, perm = oracle.csr_to_csc(c["rowptr"], c["col"],
                                                   np.array(c["val"], np.float32), c["n_cols"])
    assert colptr.tolist() == c["colptr"]
    assert perm.tolist() == c["perm"]
    assert row_t.tolist() == c["row_t"]
    assert val_t.tolist() == c["val_t"]


def test_csc_matches_scipy_and_dense():
    rng = np.random.default_rng(13)
    for g in _graphs(3):
        colptr, row_t, val_t, perm = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
        # dense A^T
        T = np.zeros((g.n_cols, g.n_rows))
        cols = np.repeat(np.arange(g.n_cols), np.diff(colptr))
        np.add.at(T, (cols, row_t), val_t.astype(np.float64))
        np.testing.assert_array_equal(T, _dense(g).T)
        # permutation and bit copies
        assert np.array_equal(np.sort(perm), np.arange(g.nnz))
        assert np.array_equal(val_t.view(np.uint32), g.val[perm].view(np.uint32))
        rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
        assert np.array_equal(row_t, rows[perm])
        assert np.all(np.diff(g.col[perm]) >= 0)
        # stability: inside a column, increasing CSR edge id
        for j in range(g.n_cols):
            seg = perm[colptr[j]:colptr[j + 1]]
            assert np.all(np.diff(seg) > 0)
    g = synth.random_csr(500, 400, rng, mean_deg=7)      # canonical (sorted, unique)
    colptr, row_t, _, _ = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
    S = sp.csr_matrix((g.val, g.col, g.rowptr), shape=(g.n_rows, g.n_cols)).tocsc()
    S.sort_indices()
    assert np.array_equal(colptr, S.indptr) and np.array_equal(row_t, S.indices)


def test_csc_double_transpose_is_identity():
    rng = np.random.default_rng(14)
    g = synth.random_csr(300, 250, rng, mean_deg=6, empty_frac=0.1)
    colptr, row_t, val_t, _ = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
    rp2, col2, val2, _ = oracle.csr_to_csc(colptr, row_t, val_t, g.n_rows)
    assert np.array_equal(rp2, g.rowptr) and np.array_equal(col2, g.col)
    assert np.array_equal(val2.view(np.uint32), g.val.view(np.uint32))


# ------------------------------------------------------------ SpMM^T

def test_spmm_t_golden_hand_example():
    with open(os.path.join(GOLDEN, "csr_dups_unsorted.json")) as f:
        c = json.load(f)
    dX, _ = oracle.spmm_t(c["rowptr"], c["col"], np.array(c["val"], np.float32),
                          np.array(c["G"], np.float32), c["n_cols"])
    assert dX.tolist() == c["dX"]


def test_spmm_t_dense_and_adjoint():
    rng = np.random.default_rng(15)
    for g in _graphs(4):
        F = 6
        X = rng.standard_normal((g.n_cols, F)).astype(np.float32)
        G = rng.standard_normal((g.n_rows, F)).astype(np.float32)
        dX, _ = oracle.spmm_t(g.rowptr, g.col, g.val, G, g.n_cols)
        np.testing.assert_allclose(dX, _dense(g).T @ G.astype(np.float64), rtol=1e-12, atol=1e-12)
        Y, _ = oracle.spmm(g.rowptr, g.col, g.val, X)
        lhs = float(np.sum(Y * G.astype(np.float64)))
        rhs = float(np.sum(X.astype(np.float64) * dX))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


def test_spmm_t_equals_spmm_on_transposed_csr_and_selection():
    rng = np.random.default_rng(16)
    g = synth.random_csr(400, 300, rng, mean_deg=5, dup=True, unsorted=True)
    G = rng.standard_normal((400, 4)).astype(np.float32)
    colptr, row_t, val_t, _ = oracle.csr_to_csc(g.rowptr, g.col, g.val, g.n_cols)
    dX, A = oracle.spmm_t(g.rowptr, g.col, g.val, G, g.n_cols)
    Y2, A2 = oracle.spmm(colptr, row_t, val_t, G)
    assert np.array_equal(dX, Y2) and np.array_equal(A, A2)   # same terms, same order
    sel = np.array([5, 299, 0, 100], dtype=np.int32)
    dXs, _ = oracle.spmm_t(g.rowptr, g.col, g.val, G, g.n_cols, cols=sel)
    assert np.array_equal(dXs, dX[sel])


# ------------------------------------------------------------ edge softmax

def _lrelu(t, slope=0.2):
    return np.where(t > 0, t, slope * t)


def test_softmax_closed_forms():
    one_row = np.array([0, 2], dtype=np.int32)
    col = np.array([0, 1], dtype=np.int32)
    # e = [0.5, 1.5] (positive branch): alpha = [1/(1+e), e/(1+e)] with e = exp(1)
    a = oracle.edge_softmax(one_row, col, np.zeros((1, 1), np.float32),
                            np.array([[0.5], [1.5]], np.float32))
    E = math.e
    assert abs(a[0, 0] - 1 / (1 + E)) < 1e-15 and abs(a[1, 0] - E / (1 + E)) < 1e-15
    # t = [-1, -2] (negative branch, slope 0.2): e = [-0.2, -0.4]
    a = oracle.edge_softmax(one_row, col, np.zeros((1, 1), np.float32),
                            np.array([[-1.0], [-2.0]], np.float32))
    w = math.exp(-0.2)
    assert abs(a[0, 0] - 1 / (1 + w)) < 1e-15
    assert abs(a[1, 0] - w / (1 + w)) < 1e-15
    # mixed signs, two heads, s_dst added: t = s_dst + s_src
    rp = np.array([0, 3], dtype=np.int32)
    c3 = np.array([0, 1, 2], dtype=np.int32)
    sd = np.array([[0.25, -1.0]], np.float32)
    ss = np.array([[0.75, 2.0], [-1.25, 1.0], [-0.25, 0.0]], np.float32)
    a = oracle.edge_softmax(rp, c3, sd, ss, slope=0.2)
    e0 = np.array([1.0, -0.2, 0.0])                 # head 0: t = [1, -1, 0]
    e1 = np.array([1.0, 0.0, -0.2])                 # head 1: t = [1, 0, -1]
    for h, e in ((0, e0), (1, e1)):
        want = np.exp(e) / np.exp(e).sum()
        np.testing.assert_allclose(a[:, h], want, rtol=1e-15)


def test_softmax_invariants_and_brute_force():
    rng = np.random.default_rng(17)
    for n in (1, 2, 5, 9, 16):
        g = synth.random_csr(n, n, rng, mean_deg=4, empty_frac=0.2)
        H = 3
        sd = rng.standard_normal((n, H)).astype(np.float32)
        ss = rng.standard_normal((n, H)).astype(np.float32)
        a = oracle.edge_softmax(g.rowptr, g.col, sd, ss, slope=0.2)
        assert np.all(a > 0)
        rows = np.repeat(np.arange(n), np.diff(g.rowptr))
        for h in range(H):
            sums = np.bincount(rows, weights=a[:, h], minlength=n)
            nonempty = np.diff(g.rowptr) > 0
            np.testing.assert_allclose(sums[nonempty], 1.0, rtol=0, atol=1e-14)
            # dense masked softmax, -inf off the pattern
            S = np.full((n, n), -np.inf)
            S[rows, g.col] = _lrelu(sd[rows, h].astype(np.float64) + ss[g.col, h].astype(np.float64))
            for i in np.flatnonzero(nonempty):
                p = np.exp(S[i] - S[i].max())
                p /= p.sum()
                np.testing.assert_allclose(a[g.rowptr[i]:g.rowptr[i + 1], h], p[g.col[g.rowptr[i]:g.rowptr[i + 1]]],
                                           rtol=1e-13)


def test_softmax_special_cases():
    rng = np.random.default_rng(18)
    g = synth.random_csr(200, 150, rng, mean_deg=6, empty_frac=0.1, dup=True)
    H = 4
    sd = rng.standard_normal((200, H)).astype(np.float32)
    d = np.diff(g.rowptr)
    rows = np.repeat(np.arange(200), d)
    # s_src == 0: all scores of a row are equal -> alpha = 1/d
    a = oracle.edge_softmax(g.rowptr, g.col, sd, np.zeros((150, H), np.float32))
    np.testing.assert_allclose(a, np.repeat(1.0 / d[rows], H).reshape(-1, H), rtol=1e-15)
    # degree-1 rows give exactly 1
    ss = rng.standard_normal((150, H)).astype(np.float32) * 30
    a = oracle.edge_softmax(g.rowptr, g.col, sd, ss)
    one = d[rows] == 1
    assert np.all(a[one] == 1.0)
    # huge scores: max subtraction keeps exp finite
    a = oracle.edge_softmax(g.rowptr, g.col, sd * 1000, ss * 100)
    assert np.all(np.isfinite(a))
    sums = np.bincount(rows, weights=a[:, 0], minlength=200)
    np.testing.assert_allclose(sums[d > 0], 1.0, atol=1e-13)
    # all-positive t: a per-row shift of s_dst shifts e and leaves alpha unchanged
    sdp = np.abs(sd) + 40.0
    a0 = oracle.edge_softmax(g.rowptr, g.col, sdp, ss / 30)
    a1 = oracle.edge_softmax(g.rowptr, g.col, sdp + 5.0, ss / 30)
    np.testing.assert_allclose(a0, a1, rtol=1e-12)


def test_softmax_selected_rows_pack_in_order():
    rng = np.random.default_rng(19)
    g = synth.random_csr(100, 80, rng, mean_deg=5, empty_frac=0.1)
    sd = rng.standard_normal((100, 2)).astype(np.float32)
    ss = rng.standard_normal((80, 2)).astype(np.float32)
    a = oracle.edge_softmax(g.rowptr, g.col, sd, ss)
    sel = np.array([7, 3, 99], dtype=np.int32)
    part = oracle.edge_softmax(g.rowptr, g.col, sd, ss, rows=sel)
    want = np.concatenate([a[g.rowptr[i]:g.rowptr[i + 1]] for i in sel])
    assert np.array_equal(part, want)


# ------------------------------------------------------------ GAT aggregate

def test_gat_dense_per_head_brute_force():
    rng = np.random.default_rng(20)
    for n, H, D in ((6, 1, 4), (11, 3, 5), (16, 2, 8)):
        g = synth.random_csr(n, n, rng, mean_deg=4, empty_frac=0.15)
        sd = rng.standard_normal((n, H)).astype(np.float32)
        ss = rng.standard_normal((n, H)).astype(np.float32)
        X = rng.standard_normal((n, H * D)).astype(np.float32)
        Y, _ = oracle.gat(g.rowptr, g.col, sd, ss, X, H, D, slope=0.2)
        rows = np.repeat(np.arange(n), np.diff(g.rowptr))
        Xh = X.reshape(n, H, D).astype(np.float64)
        for h in range(H):
            S = np.full((n, n), -np.inf)
            S[rows, g.col] = _lrelu(sd[rows, h].astype(np.float64) + ss[g.col, h].astype(np.float64))
            P = np.zeros((n, n))
            for i in range(n):
                if np.isfinite(S[i]).any():
                    P[i] = np.exp(S[i] - S[i].max())
                    P[i] /= P[i].sum()
            np.testing.assert_allclose(Y.reshape(n, H, D)[:, h, :], P @ Xh[:, h, :],
                                       rtol=1e-12, atol=1e-13)


def test_gat_reduces_to_spmm_and_mean():
    rng = np.random.default_rng(21)
    g = synth.random_csr(150, 120, rng, mean_deg=6, dup=True, empty_frac=0.1)
    X = rng.standard_normal((120, 16)).astype(np.float32)
    # H = 1 with alpha_in = edge values is the plain SpMM
    Yg, Ag = oracle.gat(g.rowptr, g.col, None, None, X, 1, 16, alpha_in=g.val.reshape(-1, 1))
    Ys, As = oracle.spmm(g.rowptr, g.col, g.val, X)
    assert np.array_equal(Yg, Ys) and np.array_equal(Ag, As)
    # s_src == 0: every head is the mean of the neighbour rows
    H, D = 4, 4
    sd = rng.standard_normal((150, H)).astype(np.float32)
    Y, _ = oracle.gat(g.rowptr, g.col, sd, np.zeros((120, H), np.float32), X, H, D)
    for i in range(150):
        b, e = g.rowptr[i], g.rowptr[i + 1]
        want = X[g.col[b:e]].astype(np.float64).mean(0) if e > b else np.zeros(16)
        np.testing.assert_allclose(Y[i], want, rtol=1e-13, atol=1e-15)


def test_gat_each_head_is_an_spmm_with_its_weights():
    rng = np.random.default_rng(22)
    g = synth.random_csr(90, 70, rng, mean_deg=5)
    H, D = 3, 2
    alpha = rng.random((g.nnz, H)).astype(np.float32)
    X = rng.standard_normal((70, H * D)).astype(np.float32)
    Y, _ = oracle.gat(g.rowptr, g.col, None, None, X, H, D, alpha_in=alpha)
    for h in range(H):
        Yh, _ = oracle.spmm(g.rowptr, g.col, alpha[:, h].copy(),
                            np.ascontiguousarray(X.reshape(70, H, D)[:, h, :]))
        assert np.array_equal(Y.reshape(90, H, D)[:, h, :], Yh)


# ------------------------------------------------------------ GSpMM mean / max

def test_gspmm_sum_is_spmm_and_mean_is_degree_normalized():
    rng = np.random.default_rng(30)
    for g in _graphs(5):
        X = rng.standard_normal((g.n_cols, 5)).astype(np.float32)
        Ys, As, _ = oracle.gspmm(g.rowptr, g.col, g.val, X, reduce="sum")
        Y0, A0 = oracle.spmm(g.rowptr, g.col, g.val, X)
        assert np.array_equal(Ys, Y0) and np.array_equal(As, A0)
        Ym, Am, arg = oracle.gspmm(g.rowptr, g.col, g.val, X, reduce="mean")
        assert arg is None
        d = np.diff(g.rowptr).astype(np.float64)
        want = (_dense(g) @ X.astype(np.float64)) / np.maximum(d, 1.0)[:, None]
        np.testing.assert_allclose(Ym, want, rtol=1e-12, atol=1e-14)
        # no edge values: the neighbour mean
        Yn, _, _ = oracle.gspmm(g.rowptr, g.col, None, X, reduce="mean")
        for i in range(g.n_rows):
            b, e = g.rowptr[i], g.rowptr[i + 1]
            w = X[g.col[b:e]].astype(np.float64).mean(0) if e > b else np.zeros(5)
            np.testing.assert_allclose(Yn[i], w, rtol=1e-13, atol=1e-15)


def test_gspmm_max_dense_masked_max():
    """max_j fl32(W_ij * X_jf) over the pattern, with numpy's float32 product and
    first-index argmax on graphs with sorted, distinct columns."""
    rng = np.random.default_rng(31)
    for n_rows, n_cols in ((40, 30), (7, 50), (60, 60)):
        g = synth.random_csr(n_rows, n_cols, rng, mean_deg=5, empty_frac=0.15)
        X = rng.standard_normal((n_cols, 6)).astype(np.float32)
        Y, A, arg = oracle.gspmm(g.rowptr, g.col, g.val, X, reduce="max")
        assert np.all(A == 0)
        Wd = np.zeros((n_rows, n_cols), np.float32)
        mask = np.zeros((n_rows, n_cols), bool)
        rows = np.repeat(np.arange(n_rows), np.diff(g.rowptr))
        Wd[rows, g.col] = g.val
        mask[rows, g.col] = True
        P = Wd[:, :, None] * X[None, :, :]                      # float32 products
        P = np.where(mask[:, :, None], P, -np.inf)
        jmax = np.argmax(P, axis=1)                             # first max in column order
        empty = ~mask.any(1)
        want = np.where(empty[:, None], 0.0, P.max(1).astype(np.float64))
        assert np.array_equal(Y, want)
        # the first maximal column of a sorted row is its first maximal edge
        want_arg = np.where(empty[:, None], -1,
                            g.rowptr[:-1, None] + np.array([[np.searchsorted(g.col[g.rowptr[i]:g.rowptr[i + 1]], jmax[i, f])
                                                             for f in range(6)] for i in range(n_rows)]))
        assert np.array_equal(arg, want_arg)


def test_gspmm_max_ties_take_the_first_edge():
    # row 0: the same column three times with equal weights -> the first edge
    rowptr = np.array([0, 3, 5], np.int32)
    col = np.array([1, 1, 1, 0, 1], np.int32)
    val = np.array([2.0, 2.0, 2.0, -1.0, -1.0], np.float32)
    X = np.array([[1.0, -3.0], [0.5, -0.25]], np.float32)
    Y, _, arg = oracle.gspmm(rowptr, col, val, X, reduce="max")
    assert Y.tolist() == [[1.0, -0.5], [-0.5, 3.0]]
    assert arg.tolist() == [[0, 0], [4, 3]]
    # no edge values: the plain neighbour max
    Y, _, arg = oracle.gspmm(rowptr, col, None, X, reduce="max")
    assert Y.tolist() == [[0.5, -0.25], [1.0, -0.25]]
    assert arg.tolist() == [[0, 0], [3, 4]]


# ------------------------------------------------------------ GSpMM compute operators

def _pattern_and_rowsum(g):
    """Dense pattern counts P (duplicates add up) and the row sums of the edge values."""
    P = np.zeros((g.n_rows, g.n_cols))
    rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
    np.add.at(P, (rows, g.col), 1.0)
    wsum = np.zeros(g.n_rows)
    np.add.at(wsum, rows, g.val.astype(np.float64))
    return P, wsum


def test_gspmm_add_sub_sum_and_mean_closed_forms():
    """sum_k (x_kf + w_k) = (P X)_if + sum_k w_k, and the same with -w for sub;
    mean divides both by the degree; Abs is the sum of |message|."""
    rng = np.random.default_rng(32)
    for g in _graphs(6):
        X = rng.standard_normal((g.n_cols, 4)).astype(np.float32)
        P, wsum = _pattern_and_rowsum(g)
        PX = P @ X.astype(np.float64)
        d = np.diff(g.rowptr).astype(np.float64)
        for op, sign in (("add", 1.0), ("sub", -1.0)):
            Y, A, _ = oracle.gspmm(g.rowptr, g.col, g.val, X, "sum", compute=op)
            np.testing.assert_allclose(Y, PX + sign * wsum[:, None], rtol=1e-12, atol=1e-12)
            Ym, Am, _ = oracle.gspmm(g.rowptr, g.col, g.val, X, "mean", compute=op)
            np.testing.assert_allclose(Ym, (PX + sign * wsum[:, None]) / np.maximum(d, 1)[:, None],
                                       rtol=1e-12, atol=1e-12)
            # error scale by brute force over the edges of each row
            for i in range(g.n_rows):
                b, e = g.rowptr[i], g.rowptr[i + 1]
                m = X[g.col[b:e]].astype(np.float64) + sign * g.val[b:e, None].astype(np.float64)
                np.testing.assert_allclose(A[i], np.abs(m).sum(0), rtol=1e-13, atol=0)
                np.testing.assert_allclose(Am[i], np.abs(m).sum(0) / max(e - b, 1), rtol=1e-13, atol=0)


def test_gspmm_copy_ignores_values():
    rng = np.random.default_rng(33)
    for g in _graphs(7):
        X = rng.standard_normal((g.n_cols, 3)).astype(np.float32)
        P, _ = _pattern_and_rowsum(g)
        Y, _, _ = oracle.gspmm(g.rowptr, g.col, g.val, X, "sum", compute="copy")
        np.testing.assert_allclose(Y, P @ X.astype(np.float64), rtol=1e-12, atol=1e-12)
        for red in ("sum", "mean", "max"):
            a = oracle.gspmm(g.rowptr, g.col, g.val, X, red, compute="copy")
            b = oracle.gspmm(g.rowptr, g.col, None, X, red, compute="mul")
            assert np.array_equal(a[0], b[0])
            assert (a[2] is None and b[2] is None) or np.array_equal(a[2], b[2])


def test_gspmm_max_add_dense_masked_max():
    """max_j fl32(X_jf + W_ij) over the pattern with numpy's float32 sum."""
    rng = np.random.default_rng(34)
    for n_rows, n_cols in ((30, 40), (64, 20)):
        g = synth.random_csr(n_rows, n_cols, rng, mean_deg=6, empty_frac=0.2)
        X = rng.standard_normal((n_cols, 5)).astype(np.float32)
        rows = np.repeat(np.arange(n_rows), np.diff(g.rowptr))
        mask = np.zeros((n_rows, n_cols), bool)
        mask[rows, g.col] = True
        empty = ~mask.any(1)
        for op, sign in (("add", 1), ("sub", -1)):
            Wd = np.zeros((n_rows, n_cols), np.float32)
            Wd[rows, g.col] = g.val
            M = X[None, :, :] + np.float32(sign) * Wd[:, :, None]       # float32 sums
            M = np.where(mask[:, :, None], M, -np.inf)
            Y, _, arg = oracle.gspmm(g.rowptr, g.col, g.val, X, "max", compute=op)
            assert np.array_equal(Y, np.where(empty[:, None], 0.0, M.max(1).astype(np.float64)))
            jmax = np.argmax(M, axis=1)
            got_cols = np.where(arg >= 0, g.col[np.maximum(arg, 0)], -1)
            assert np.array_equal(got_cols, np.where(empty[:, None], -1, jmax))


def test_gspmm_compute_hand_example():
    # row 0: edges (col 1, w 2), (col 0, w -1); row 1 empty; X = [[1, -3], [0.5, -0.25]]
    rowptr = np.array([0, 2, 2], np.int32)
    col = np.array([1, 0], np.int32)
    val = np.array([2.0, -1.0], np.float32)
    X = np.array([[1.0, -3.0], [0.5, -0.25]], np.float32)
    Y, A, _ = oracle.gspmm(rowptr, col, val, X, "sum", compute="add")
    assert Y.tolist() == [[2.5 + 0.0, 1.75 - 4.0], [0.0, 0.0]]
    assert A.tolist() == [[2.5, 1.75 + 4.0], [0.0, 0.0]]
    Y, _, arg = oracle.gspmm(rowptr, col, val, X, "max", compute="sub")
    # messages: edge 0 -> (0.5-2, -0.25-2) = (-1.5, -2.25); edge 1 -> (1+1, -3+1) = (2, -2)
    assert Y.tolist() == [[2.0, -2.0], [0.0, 0.0]]
    assert arg.tolist() == [[1, 1], [-1, -1]]
    Y, _, _ = oracle.gspmm(rowptr, col, val, X, "mean", compute="sub")
    assert Y.tolist() == [[(-1.5 + 2.0) / 2, (-2.25 - 2.0) / 2], [0.0, 0.0]]


# ------------------------------------------------------------ GAT backward

def _dense_heads(g, H, D, Xf, dYf):
    return Xf.reshape(g.n_cols, H, D).astype(np.float64), dYf.reshape(g.n_rows, H, D).astype(np.float64)


def test_sddmm_dot_dense():
    """out[k,h] = (P_h Q_h^T)[i, col[k]] for every edge, duplicates included."""
    rng = np.random.default_rng(40)
    for g in _graphs(8):
        H, D = 3, 5
        P = rng.standard_normal((g.n_rows, H * D)).astype(np.float32)
        Q = rng.standard_normal((g.n_cols, H * D)).astype(np.float32)
        out, ab = oracle.sddmm_dot(g.rowptr, g.col, P, Q, H, D)
        rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
        for h in range(H):
            M = P.reshape(-1, H, D)[:, h, :].astype(np.float64) @ Q.reshape(-1, H, D)[:, h, :].astype(np.float64).T
            Ma = np.abs(P.reshape(-1, H, D)[:, h, :].astype(np.float64)) @ np.abs(Q.reshape(-1, H, D)[:, h, :].astype(np.float64)).T
            np.testing.assert_allclose(out[:, h], M[rows, g.col], rtol=1e-13, atol=1e-13)
            np.testing.assert_allclose(ab[:, h], Ma[rows, g.col], rtol=1e-13, atol=1e-13)
        # selected rows pack their edges in list order
        sel = np.array([g.n_rows - 1, 0], np.int32)
        o2, _ = oracle.sddmm_dot(g.rowptr, g.col, P, Q, H, D, rows=sel)
        idx = np.concatenate([np.arange(g.rowptr[r], g.rowptr[r + 1]) for r in sel])
        assert np.array_equal(o2, out[idx])


def test_gat_backward_hand_example():
    # one row, two edges, H = D = 1; alpha is an input of the backward, chosen by hand
    rowptr = np.array([0, 2], np.int32)
    col = np.array([0, 1], np.int32)
    X = np.array([[2.0], [3.0]], np.float32)
    dY = np.array([[1.0]], np.float32)
    s_dst = np.array([[0.0]], np.float32)
    s_src = np.array([[1.0], [-1.0]], np.float32)
    alpha = np.array([[0.75], [0.25]], np.float32)
    r = oracle.gat_backward(rowptr, col, s_dst, s_src, alpha, X, dY, 1, 1, slope=0.2)
    assert r["dalpha"].ravel().tolist() == [2.0, 3.0]
    # c = 0.75*2 + 0.25*3 = 2.25; t = (1, -1) -> f = (1, 0.2)
    assert r["dscore"].ravel().tolist() == [0.75 * (2 - 2.25), 0.2 * 0.25 * (3 - 2.25)]
    assert r["ds_dst"].ravel().tolist() == [0.75 * (2 - 2.25) + 0.2 * 0.25 * (3 - 2.25)]
    assert r["ds_src"].ravel().tolist() == [0.75 * (2 - 2.25), 0.2 * 0.25 * (3 - 2.25)]
    assert r["dX"].ravel().tolist() == [0.75, 0.25]


def _softmax_forward_dense(g, sd, ss, X, H, D, slope):
    """Dense fp64 GAT forward on a graph without duplicate edges."""
    mask = np.zeros((g.n_rows, g.n_cols), bool)
    rows = np.repeat(np.arange(g.n_rows), np.diff(g.rowptr))
    mask[rows, g.col] = True
    Y = np.zeros((g.n_rows, H, D))
    A = np.zeros((H, g.n_rows, g.n_cols))
    for h in range(H):
        t = sd[:, h, None] + ss[None, :, h]
        e = np.where(t > 0, t, slope * t)
        e = np.where(mask, e, -np.inf)
        m = e.max(1, keepdims=True)
        m[~np.isfinite(m)] = 0.0
        p = np.where(mask, np.exp(e - m), 0.0)
        z = p.sum(1, keepdims=True)
        a = np.divide(p, z, out=np.zeros_like(p), where=z > 0)
        A[h] = a
        Y[:, h, :] = a @ X[:, h, :]
    return Y, A


def test_gat_backward_matches_finite_differences():
    """ds_dst and ds_src against central differences of a dense fp64 forward,
    dX against the transposed dense attention, dalpha against the dense SDDMM."""
    rng = np.random.default_rng(41)
    H, D, slope = 2, 3, 0.2
    for n in (6, 11, 16):
        g = synth.random_csr(n, n, rng, mean_deg=3, empty_frac=0.1)
        while True:
            sd = rng.standard_normal((n, H)).astype(np.float32)
            ss = rng.standard_normal((n, H)).astype(np.float32)
            t = sd.astype(np.float64)[np.repeat(np.arange(n), np.diff(g.rowptr))] + ss.astype(np.float64)[g.col]
            if np.abs(t).min() > 1e-2:      # keep clear of the LeakyReLU kink
                break
        X = rng.standard_normal((n, H * D)).astype(np.float32)
        dY = rng.standard_normal((n, H * D)).astype(np.float32)
        Xd, dYd = _dense_heads(g, H, D, X, dY)
        _, A = _softmax_forward_dense(g, sd.astype(np.float64), ss.astype(np.float64), Xd, H, D, slope)
        rows = np.repeat(np.arange(n), np.diff(g.rowptr))
        alpha = np.stack([A[h][rows, g.col] for h in range(H)], 1).astype(np.float32)
        r = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, X, dY, H, D, slope=slope)

        def loss(sd64, ss64):
            Y, _ = _softmax_forward_dense(g, sd64, ss64, Xd, H, D, slope)
            return float(np.sum(Y * dYd))

        eps = 1e-6
        base_d, base_s = sd.astype(np.float64), ss.astype(np.float64)
        fd_dst = np.zeros((n, H))
        fd_src = np.zeros((n, H))
        for i in range(n):
            for h in range(H):
                p, m = base_d.copy(), base_d.copy()
                p[i, h] += eps
                m[i, h] -= eps
                fd_dst[i, h] = (loss(p, base_s) - loss(m, base_s)) / (2 * eps)
                p, m = base_s.copy(), base_s.copy()
                p[i, h] += eps
                m[i, h] -= eps
                fd_src[i, h] = (loss(base_d, p) - loss(base_d, m)) / (2 * eps)
        # alpha is rounded to fp32 for the backward: agreement to ~1e-6 of the scale
        scale = np.abs(fd_dst).max() + np.abs(fd_src).max() + 1.0
        assert np.abs(r["ds_dst"] - fd_dst).max() <= 2e-6 * scale
        assert np.abs(r["ds_src"] - fd_src).max() <= 2e-6 * scale
        for h in range(H):
            dXh = A[h].astype(np.float32).astype(np.float64).T @ dYd[:, h, :]
            np.testing.assert_allclose(r["dX"].reshape(n, H, D)[:, h, :], dXh, rtol=1e-12, atol=1e-12)
            M = dYd[:, h, :] @ Xd[:, h, :].T
            np.testing.assert_allclose(r["dalpha"][:, h], M[rows, g.col], rtol=1e-12, atol=1e-12)


def test_gat_backward_invariants():
    rng = np.random.default_rng(42)
    H, D = 3, 4
    for g in _graphs(9):
        sd = rng.standard_normal((g.n_rows, H)).astype(np.float32)
        ss = rng.standard_normal((g.n_cols, H)).astype(np.float32)
        alpha = oracle.edge_softmax(g.rowptr, g.col, sd, ss, slope=1.0).astype(np.float32)
        X = rng.standard_normal((g.n_cols, H * D)).astype(np.float32)
        dY = rng.standard_normal((g.n_rows, H * D)).astype(np.float32)
        # slope 1: the softmax backward sums to zero over each row (sum alpha = 1)
        r = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, X, dY, H, D, slope=1.0)
        assert np.all(np.abs(r["ds_dst"]) <= 1e-6 * r["ds_dst_abs"] + 1e-300)
        # degree-1 rows: alpha = 1 exactly, so their score gradients are exactly 0
        d = np.diff(g.rowptr)
        one = np.flatnonzero(np.repeat(d, d) == 1)
        assert np.all(r["dscore"][one] == 0.0)
        # adjoint identity for dX with the forward aggregation at fixed weights
        Z = rng.standard_normal((g.n_cols, H * D)).astype(np.float32)
        Yz, _ = oracle.gat(g.rowptr, g.col, None, None, Z, H, D, alpha_in=alpha)
        lhs = float(np.sum(r["dX"] * Z.astype(np.float64)))
        rhs = float(np.sum(Yz * dY.astype(np.float64)))
        assert abs(lhs - rhs) <= 1e-11 * (np.abs(r["dX"]).sum() * np.abs(Z).max() + 1.0)
        # dalpha is the dot-product SDDMM of dY and X
        dot, _ = oracle.sddmm_dot(g.rowptr, g.col, dY, X, H, D)
        assert np.array_equal(dot, r["dalpha"])
        # row and column selections give the same values
        sel = np.array([g.n_rows - 1, 0], np.int32)
        csel = np.array([g.n_cols - 1, 0], np.int32)
        r2 = oracle.gat_backward(g.rowptr, g.col, sd, ss, alpha, X, dY, H, D, slope=1.0, rows=sel, cols=csel)
        assert np.array_equal(r2["ds_dst"], r["ds_dst"][sel])
        assert np.array_equal(r2["ds_src"], r["ds_src"][csel])
        assert np.array_equal(r2["dX"], r["dX"][csel])
        idx = np.concatenate([np.arange(g.rowptr[x], g.rowptr[x + 1]) for x in sel])
        assert np.array_equal(r2["dscore"], r["dscore"][idx])


# ------------------------------------------------------------ dense layers and 2-layer models

def _bf16(x):
    return synth.f32_to_bf16_bits(np.asarray(x, np.float32))


def _dec(bits):
    return oracle.decode(bits, oracle.BF16)


def test_linear_against_numpy():
    rng = np.random.default_rng(50)
    for n, k, m in ((7, 5, 3), (33, 602, 41), (1, 16, 128)):
        X, W = _bf16(rng.standard_normal((n, k))), _bf16(rng.standard_normal((m, k)))
        b = rng.standard_normal(m).astype(np.float32)
        for act in ("none", "relu", "elu"):
            Y, A = oracle.linear(X, W, b, act, x_dtype=oracle.BF16, w_dtype=oracle.BF16)
            pre = _dec(X) @ _dec(W).T + b.astype(np.float64)
            want = {"none": pre, "relu": np.maximum(pre, 0.0), "elu": np.where(pre > 0, pre, np.expm1(pre))}[act]
            np.testing.assert_allclose(Y, want, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(A, np.abs(_dec(X)) @ np.abs(_dec(W)).T + np.abs(b), rtol=1e-12)


def test_epilogue_closed_forms():
    v = np.array([[-1.0, 0.0, 2.0]])
    assert oracle.epilogue(v.copy(), None, "relu").tolist() == [[0.0, 0.0, 2.0]]
    e = oracle.epilogue(v.copy(), None, "elu")
    assert e[0, 0] == np.expm1(-1.0) and e[0, 1] == 0.0 and e[0, 2] == 2.0
    b = np.array([1.0, -1.0, 0.5], np.float32)
    assert oracle.epilogue(v.copy(), b, "none").tolist() == [[0.0, -1.0, 2.5]]


def test_head_scores_against_numpy():
    rng = np.random.default_rng(51)
    n, H, D = 40, 3, 7
    Z = _bf16(rng.standard_normal((n, H * D)))
    a_s, a_d = rng.standard_normal((H, D)).astype(np.float32), rng.standard_normal((H, D)).astype(np.float32)
    ss, sd, sa, da = oracle.head_scores(Z, a_s, a_d, H, D, z_dtype=oracle.BF16)
    Zd = _dec(Z).reshape(n, H, D)
    np.testing.assert_allclose(ss, np.einsum("nhd,hd->nh", Zd, a_s.astype(np.float64)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sd, np.einsum("nhd,hd->nh", Zd, a_d.astype(np.float64)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sa, np.einsum("nhd,hd->nh", np.abs(Zd), np.abs(a_s)), rtol=1e-12)
    np.testing.assert_allclose(da, np.einsum("nhd,hd->nh", np.abs(Zd), np.abs(a_d)), rtol=1e-12)


def _mlp_params(rng, k, hid, out):
    return dict(W1=_bf16(rng.standard_normal((hid, k)) * 0.3), b1=rng.standard_normal(hid).astype(np.float32),
                W2=_bf16(rng.standard_normal((out, hid)) * 0.3), b2=rng.standard_normal(out).astype(np.float32))


def test_gcn_forward_identity_graph_is_an_mlp():
    """With A = I the model is relu(X W1^T + b1) W2^T + b2, activations stored in bf16."""
    rng = np.random.default_rng(52)
    n, k, hid, out = 30, 12, 16, 5
    rowptr = np.arange(n + 1, dtype=np.int32)
    col = np.arange(n, dtype=np.int32)
    X = _bf16(rng.standard_normal((n, k)))
    p = _mlp_params(rng, k, hid, out)
    Y, E = oracle.gcn_forward(rowptr, col, None, X, p)
    Z1 = _dec(oracle.round_to(_dec(X) @ _dec(p["W1"]).T, oracle.BF16))
    H1 = _dec(oracle.round_to(np.maximum(Z1 + p["b1"], 0.0), oracle.BF16))
    Z2 = _dec(oracle.round_to(H1 @ _dec(p["W2"]).T, oracle.BF16))
    np.testing.assert_allclose(Y, Z2 + p["b2"], rtol=1e-12, atol=1e-12)
    assert np.all(np.abs(Y) <= E * (1 + 2 ** -6))
    # selected output rows
    sel = np.array([n - 1, 3], np.int32)
    Ys, Es = oracle.gcn_forward(rowptr, col, None, X, p, rows=sel)
    assert np.array_equal(Ys, Y[sel]) and np.array_equal(Es, E[sel])


def test_gcn_forward_dense_graph():
    """On a small irregular graph: the dense A applied between the stored layers."""
    rng = np.random.default_rng(53)
    g = synth.random_csr(25, 25, rng, mean_deg=4, empty_frac=0.1)
    X = _bf16(rng.standard_normal((25, 10)))
    p = _mlp_params(rng, 10, 8, 3)
    Y, E = oracle.gcn_forward(g.rowptr, g.col, g.val, X, p)
    A = _dense(g)
    Z1 = _dec(oracle.round_to(_dec(X) @ _dec(p["W1"]).T, oracle.BF16))
    H1 = _dec(oracle.round_to(np.maximum(A @ Z1 + p["b1"], 0.0), oracle.BF16))
    Z2 = _dec(oracle.round_to(H1 @ _dec(p["W2"]).T, oracle.BF16))
    np.testing.assert_allclose(Y, A @ Z2 + p["b2"], rtol=1e-11, atol=1e-11)


def test_gat_forward_zero_attention_is_a_mean():
    """With zero attention vectors every score is 0: each layer averages its
    neighbours' stored features (then bias, ELU on the first layer)."""
    rng = np.random.default_rng(54)
    g = synth.random_csr(25, 25, rng, mean_deg=4, empty_frac=0.1)
    n, k, H, D, C = 25, 10, 2, 4, 3
    X = _bf16(rng.standard_normal((n, k)))
    p = dict(W1=_bf16(rng.standard_normal((H * D, k)) * 0.3), a_src1=np.zeros((H, D), np.float32),
             a_dst1=np.zeros((H, D), np.float32), b1=rng.standard_normal(H * D).astype(np.float32),
             W2=_bf16(rng.standard_normal((C, H * D)) * 0.3), a_src2=np.zeros((1, C), np.float32),
             a_dst2=np.zeros((1, C), np.float32), b2=rng.standard_normal(C).astype(np.float32))
    Y, E = oracle.gat_forward(g.rowptr, g.col, X, p)
    counts = np.zeros((n, n))
    rows = np.repeat(np.arange(n), np.diff(g.rowptr))
    np.add.at(counts, (rows, g.col), 1.0)
    deg = counts.sum(1, keepdims=True)
    M = np.divide(counts, deg, out=np.zeros_like(counts), where=deg > 0)
    Z1 = _dec(oracle.round_to(_dec(X) @ _dec(p["W1"]).T, oracle.BF16))
    pre = M @ Z1 + p["b1"]
    H1 = _dec(oracle.round_to(np.where(pre > 0, pre, np.expm1(pre)), oracle.BF16))
    Z2 = _dec(oracle.round_to(H1 @ _dec(p["W2"]).T, oracle.BF16))
    np.testing.assert_allclose(Y, M @ Z2 + p["b2"], rtol=1e-11, atol=1e-11)
    assert np.all(np.abs(Y) <= E * (1 + 2 ** -6))


# ------------------------------------------------------------ activation compression codec

def test_philox_known_answers():
    kat = json.load(open(os.path.join(GOLDEN, "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        out = oracle.philox4x32_10([int(x, 16) for x in v["counter"]], [int(x, 16) for x in v["key"]])
        assert [int(x) for x in out] == [int(x, 16) for x in v["out"]]


def test_codec_bit_planes_hand_example():
    # codes j % 4 on an exact grid (m = 0, M = 3, s = r = 1): the uniform never moves them
    x = (np.arange(64) % 4).astype(np.float32)[None, :]
    codes, stats = oracle.act_compress(x, 2, 64, seed=123)
    assert stats.tolist() == [0.0, 1.0]
    assert codes.tolist() == [0xAAAAAAAAAAAAAAAA, 0xCCCCCCCCCCCCCCCC]
    assert np.array_equal(oracle.act_decompress(codes, stats, 1, 64, 2, 64), x)


def test_codec_exact_grid_and_constant_groups():
    # 8 bits, values m + j / 16: s = 16 and r = 1/16 exactly, every value recovered
    x = (np.arange(256, dtype=np.float32) / 16.0 - 3.0)[None, :]
    codes, stats = oracle.act_compress(x, 8, 256, seed=9)
    assert np.array_equal(oracle.act_decompress(codes, stats, 1, 256, 8, 256), x)
    # a constant group: every code 0, decoded exactly
    c = np.full((3, 128), 1.25, np.float32)
    codes, stats = oracle.act_compress(c, 3, 64, seed=1)
    assert not codes.any() and np.array_equal(oracle.act_decompress(codes, stats, 3, 128, 3, 64), c)


def test_codec_decoder_rounds_once():
    """The decoded value is fma(q, r, m): q * r + m rounded once to fp32 (the codec's definition).
    Hand example where one rounding and two roundings differ: m = -3, r = 1 + 2^-23 (the fp32
    just above 1), 2-bit codes 0, 1, 2, 3 on features 0..3 (bit planes 0b1010 and 0b1100).
    Exactly: q r + m = -3, -2 + 2^-23, -1 + 2^-22 and 3 * 2^-23, each an fp32 value, so the
    single rounding returns them unchanged.  Rounding q r first would give 3 r = 3 + 3 * 2^-23
    -> 3 + 2^-21 (a tie between 3 + 2^-22 and 3 + 2^-21, broken to the even significand), and
    then 2^-21 instead of 3 * 2^-23 for code 3.  Features 4..63 have code 0 and decode to m."""
    r = np.frombuffer(np.uint32(0x3F800001).tobytes(), np.float32)[0]
    stats = np.array([-3.0, r], np.float32)
    codes = np.array([0b1010, 0b1100], np.uint64)        # plane 0, plane 1 of features 0..63
    y = oracle.act_decompress(codes, stats, 1, 64, 2, 64)[0]
    want = [-3.0, -2.0 + 2.0 ** -23, -1.0 + 2.0 ** -22, 3.0 * 2.0 ** -23]
    assert [float(v) for v in y[:4]] == want
    assert float(y[3]) != 2.0 ** -21
    assert np.all(y[4:] == np.float32(-3.0))


from codec_cases import codec_uniform as _codec_uniform  # noqa: E402


def test_codec_quantizer_rounds_once():
    """The code is floor(fma(x - m, s, u)): (x - m) s + u rounded once to fp32.  Constructed case
    (1 bit, one group: x at feature 0, the maximum M at feature 1, zeros elsewhere, so m = 0 and
    s = fl(1 / M)): with u > 1/2 and T = 1 - 2^-25 - u (an fp32 value on the 2^-25 grid of
    [1/4, 1/2)), pick x so that the exact product P = x s lies strictly within 2^-26 below T.
    Then P + u lies in (1 - 3 2^-26, 1 - 2 2^-26), whose nearest fp32 value is 1 - 2^-24, so the
    single rounding gives code 0; rounding P first gives exactly T, then T + u = 1 - 2^-25, a tie
    broken to 1.0, and code 1."""
    import struct
    f32 = lambda v: struct.unpack("<f", struct.pack("<f", float(v)))[0]   # noqa: E731

    def neighbours(v, k):
        b = struct.unpack("<I", struct.pack("<f", v))[0]
        return [struct.unpack("<f", struct.pack("<I", b + d))[0] for d in range(-k, k + 1)]

    for seed in range(1, 200):
        u = _codec_uniform(seed, 0)
        if not Fraction(1, 2) < u <= Fraction(3, 4):
            continue
        T = 1 - Fraction(1, 1 << 25) - u
        for M in (3.0, 5.0, 7.0, 9.0, 11.0, 13.0):
            s = f32(1.0 / M)
            for x in neighbours(f32(float(T) / s), 64):
                P = Fraction(x) * Fraction(s)
                if 0 < x <= M and T - Fraction(1, 1 << 26) < P < T:
                    row = np.zeros((1, 64), np.float32)
                    row[0, 0], row[0, 1] = x, M
                    codes, stats = oracle.act_compress(row, 1, 64, seed=seed)
                    assert float(stats[0]) == 0.0 and float(stats[1]) == M
                    # rounding the product first would give code 1 (the test is sensitive)
                    two = np.float32(np.float32(x) * np.float32(s)) + np.float32(float(u))
                    assert np.floor(two) == 1.0
                    assert int(codes[0]) & 1 == 0, "code 0 expected from a single rounding"
                    assert int(codes[0]) >> 1 & 1 == 1   # feature 1 (= M): s M rounds to 1
                    return
    raise AssertionError("no constructed case found")


@pytest.mark.parametrize("F", [200, 256])
def test_codec_codes_follow_the_uniform_of_their_flat_index(F):
    """Each code takes the uniform of its own flat index e = i F + f (constructed in
    codec_cases.flat_index_case): any other word, counter, index or resolution of u moves some
    probe across 1.  Three rows of whole groups or of three groups and a ragged one, all four
    words of a Philox block."""
    from codec_cases import flat_index_case
    n, G, seed = 3, 64, 0x5EED0001F00D
    x, want = flat_index_case(seed, n, F, G)
    codes, stats = oracle.act_compress(x, 1, G, seed=seed)
    assert np.all(stats[0::2] == 0.0) and np.all(stats[1::2] == 1.0)
    assert np.array_equal(oracle.act_decompress(codes, stats, n, F, 1, G), want)
    assert 0 < want.sum() < want.size


@pytest.mark.parametrize("tail", [0, 8])
def test_codec_code_never_exceeds_the_top_level(tail):
    """The code is clamped to 2^b - 1 (constructed in codec_cases.clamp_case, where 255 + u
    rounds to 256; as bit planes, 256 would read back as 0)."""
    from codec_cases import clamp_case
    seed = 11
    x, e, want = clamp_case(seed, tail)
    F = x.shape[1]
    codes, stats = oracle.act_compress(x, 8, 64, seed=seed)
    g = e // 64
    assert float(stats[2 * g]) == 0.0 and float(stats[2 * g + 1]) == 1.0
    assert np.array_equal(oracle.act_decompress(codes, stats, 1, F, 8, 64), want)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_codec_error_bound_ragged_rows(bits):
    """|x' - x| < one step of the group, codes past the end of a ragged row are 0."""
    rng = np.random.default_rng(60 + bits)
    n, F, G = 17, 100, 64
    x = rng.standard_normal((n, F)).astype(np.float32)
    codes, stats = oracle.act_compress(x, bits, G, seed=77)
    y = oracle.act_decompress(codes, stats, n, F, bits, G)
    ng = 2
    step = stats[1::2].reshape(n, ng)
    per_elem = np.concatenate([np.repeat(step[:, :1], 64, 1), np.repeat(step[:, 1:], F - 64, 1)], 1)
    assert np.all(np.abs(y - x) <= per_elem * (1 + 1e-5) + 1e-7)
    w = codes.reshape(n, ng, 1, bits)
    assert not np.any(w[:, 1, 0, :] >> np.uint64(36))       # 36 valid codes in the second group
    mins = stats[0::2].reshape(n, ng)
    assert np.array_equal(mins[:, 0], x[:, :64].min(1)) and np.array_equal(mins[:, 1], x[:, 64:].min(1))


def test_codec_stochastic_rounding_is_unbiased():
    """The mean of the decoded values over many seeds converges to x (2 bits)."""
    rng = np.random.default_rng(61)
    x = rng.standard_normal((1, 64)).astype(np.float32)
    acc = np.zeros((1, 64))
    trials = 400
    for seed in range(trials):
        codes, stats = oracle.act_compress(x, 2, 64, seed=seed)
        acc += oracle.act_decompress(codes, stats, 1, 64, 2, 64)
    step = float(stats[1])
    # each decode is within one step, so its variance is at most step^2 / 4
    assert np.max(np.abs(acc / trials - x)) <= 5 * (step / 2) / np.sqrt(trials)
    # and the seed matters
    c1, _ = oracle.act_compress(x, 2, 64, seed=1)
    c2, _ = oracle.act_compress(x, 2, 64, seed=2)
    assert not np.array_equal(c1, c2)
