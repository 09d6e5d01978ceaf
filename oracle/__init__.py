"""CPU oracle for the sparse GNN operators of CogDL (arxiv 2103.00959, section 2.2).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only users.  The product library never imports,
links or runs anything here, and this package imports nothing from it.

Thin numpy/ctypes wrapper over ``oracle.c`` (plain C, fp64 arithmetic); every
function follows the definition cited in the C source.  Inputs are numpy
arrays; outputs are float64 arrays (values before the final rounding) plus the
forward-error scale ``Abs`` where applicable.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32, BF16, F16 = 0, 1, 2
ROW_SPLIT, NEIGHBOR_GROUP = 1, 2

_lib = None


def build() -> str:
    """Compile oracle.c with gcc (no fast-math, so fp64 sums stay in order)."""
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_round.argtypes = [P, i64, i32, P]
    lib.oracle_decode.argtypes = [P, i64, i32, P]
    lib.oracle_balance_mode.argtypes = [i32, i64, P]
    lib.oracle_neighbor_groups.argtypes = [i32, P, i32, i32, P]
    lib.oracle_neighbor_groups.restype = i64
    lib.oracle_spmm.argtypes = [i32, i32, i64, P, P, P, i32, P, i32, i32, P, P, P]
    lib.oracle_gspmm.argtypes = [i32, i32, i64, P, P, P, i32, P, i32, i32, i32, i32, P, P, P, P]
    lib.oracle_csr_to_csc.argtypes = [i32, i32, i64, P, P, P, P, P, P, P]
    lib.oracle_spmm_t.argtypes = [i32, i32, i64, P, P, P, i32, P, i32, i32, P, P, P]
    lib.oracle_edge_softmax.argtypes = [i32, i32, i64, P, P, i32, P, P, dbl, i32, P, P]
    lib.oracle_gat.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, dbl, P, P, i32, i32, P, P, P]
    lib.oracle_gat_backward.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, dbl, P, P, i32, P, i32,
                                        i32, P, P, P, P, P, P, P, i32, P, P, P, P, P]
    lib.oracle_sddmm_dot.argtypes = [i32, i32, i64, P, P, i32, i32, P, i32, P, i32, i32, P, P, P]
    lib.oracle_epilogue.argtypes = [i64, i32, P, i32, P]
    lib.oracle_linear.argtypes = [i64, i32, i32, P, i32, P, i32, P, i32, P, P]
    lib.oracle_head_scores.argtypes = [i64, i32, i32, P, i32, P, P, P, P, P, P]
    lib.oracle_philox4x32_10.argtypes = [P, P, P]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_act_compress.argtypes = [i64, i32, P, i32, i32, i32, ctypes.c_uint64, P, P]
    lib.oracle_act_decompress.argtypes = [i64, i32, i32, i32, P, P, P]
    _lib = lib
    return lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def _x_code(x: np.ndarray, x_dtype: int | None) -> int:
    if x_dtype is not None:
        return x_dtype
    if x.dtype == np.float32:
        return F32
    raise ValueError("16-bit inputs are passed as uint16 bit patterns with an explicit dtype code")


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with {rc}")


def set_threads(n: int) -> None:
    """Thread count for the row-parallel loops (results do not depend on it)."""
    os.environ["OMP_NUM_THREADS"] = str(n)
    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))
    except OSError:
        pass


def round_to(values: np.ndarray, dtype: int) -> np.ndarray:
    """Round float64 values to fp32 / bf16 / fp16 (nearest, ties to even) directly from
    double.  Returns float32 for F32 and uint16 bit patterns otherwise."""
    v = _c(values, np.float64).ravel()
    out = np.empty(v.size, dtype=np.float32 if dtype == F32 else np.uint16)
    _check(_load().oracle_round(_p(v), v.size, dtype, _p(out)), "round")
    return out.reshape(np.shape(values))


def decode(bits: np.ndarray, dtype: int) -> np.ndarray:
    """Exact float64 value of stored fp32 / bf16 / fp16 data."""
    b = np.ascontiguousarray(bits)
    out = np.empty(b.size, dtype=np.float64)
    _check(_load().oracle_decode(_p(b), b.size, dtype, _p(out)), "decode")
    return out.reshape(b.shape)


def balance_mode(rowptr: np.ndarray, nnz: int) -> int:
    rp = _c(rowptr, np.int32)
    return _load().oracle_balance_mode(rp.size - 1, nnz, _p(rp))


def neighbor_groups(rowptr: np.ndarray, group_size: int, mode: int) -> np.ndarray:
    """(row, begin, end) slices of at most group_size edges, in row order."""
    rp = _c(rowptr, np.int32)
    lib = _load()
    n = lib.oracle_neighbor_groups(rp.size - 1, _p(rp), group_size, mode, None)
    if n < 0:
        raise ValueError("bad neighbor-group arguments")
    out = np.empty((n, 3), dtype=np.int32)
    lib.oracle_neighbor_groups(rp.size - 1, _p(rp), group_size, mode, _p(out))
    return out


def spmm(rowptr, col, val, X, n_cols=None, x_dtype=None, rows=None):
    """Y = A X (Eq. 1, sum of products).  Returns (Y, Abs) in float64."""
    rp, cl, vl = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    X = np.ascontiguousarray(X)
    n_rows = rp.size - 1
    n_cols = X.shape[0] if n_cols is None else n_cols
    F = int(np.prod(X.shape[1:])) if X.ndim > 1 else 1
    sel = _c(rows, np.int32)
    n_out = n_rows if sel is None else sel.size
    Y = np.empty((n_out, F), dtype=np.float64)
    A = np.empty((n_out, F), dtype=np.float64)
    rc = _load().oracle_spmm(n_rows, n_cols, int(rp[-1]) if n_rows else 0, _p(rp), _p(cl), _p(vl),
                             F, _p(X), _x_code(X, x_dtype), 0 if sel is None else sel.size,
                             _p(sel), _p(Y), _p(A))
    _check(rc, "spmm")
    return Y, A


REDUCE = {"sum": 0, "mean": 1, "max": 2}
COMPUTE = {"mul": 0, "add": 1, "sub": 2, "copy": 3}


def gspmm(rowptr, col, val, X, reduce="sum", n_cols=None, x_dtype=None, rows=None, compute="mul"):
    """Eq. 1 with a sum / mean / max reduce and a mul / add / sub / copy message.
    Returns (Y, Abs, arg); arg is the first edge attaining the max (-1 for empty
    rows), None for sum / mean."""
    rp, cl, vl = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    X = np.ascontiguousarray(X)
    n_rows = rp.size - 1
    n_cols = X.shape[0] if n_cols is None else n_cols
    F = int(np.prod(X.shape[1:])) if X.ndim > 1 else 1
    sel = _c(rows, np.int32)
    n_out = n_rows if sel is None else sel.size
    Y = np.empty((n_out, F), dtype=np.float64)
    A = np.empty((n_out, F), dtype=np.float64)
    arg = np.empty((n_out, F), dtype=np.int32) if reduce == "max" else None
    rc = _load().oracle_gspmm(n_rows, n_cols, int(rp[-1]) if n_rows else 0, _p(rp), _p(cl), _p(vl),
                              F, _p(X), _x_code(X, x_dtype), REDUCE[reduce], COMPUTE[compute],
                              0 if sel is None else sel.size, _p(sel), _p(Y), _p(A), _p(arg))
    _check(rc, "gspmm")
    return Y, A, arg


def csr_to_csc(rowptr, col, val, n_cols):
    """Stable transpose. Returns (colptr, row_t, val_t, perm)."""
    rp, cl, vl = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    nnz = int(rp[-1]) if rp.size > 1 else 0
    colptr = np.empty(n_cols + 1, dtype=np.int32)
    row_t = np.empty(nnz, dtype=np.int32)
    perm = np.empty(nnz, dtype=np.int32)
    val_t = None if vl is None else np.empty(nnz, dtype=np.float32)
    rc = _load().oracle_csr_to_csc(rp.size - 1, n_cols, nnz, _p(rp), _p(cl), _p(vl), _p(colptr),
                                   _p(row_t), _p(val_t), _p(perm))
    _check(rc, "csr_to_csc")
    return colptr, row_t, val_t, perm


def spmm_t(rowptr, col, val, G, n_cols, g_dtype=None, cols=None):
    """dX = A^T G from the CSR of A.  Returns (dX, Abs) in float64."""
    rp, cl, vl = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    G = np.ascontiguousarray(G)
    F = int(np.prod(G.shape[1:])) if G.ndim > 1 else 1
    sel = _c(cols, np.int32)
    n_out = n_cols if sel is None else sel.size
    dX = np.empty((n_out, F), dtype=np.float64)
    A = np.empty((n_out, F), dtype=np.float64)
    nnz = int(rp[-1]) if rp.size > 1 else 0
    rc = _load().oracle_spmm_t(rp.size - 1, n_cols, nnz, _p(rp), _p(cl), _p(vl), F, _p(G),
                               _x_code(G, g_dtype), 0 if sel is None else sel.size, _p(sel),
                               _p(dX), _p(A))
    _check(rc, "spmm_t")
    return dX, A


def edge_softmax(rowptr, col, s_dst, s_src, slope=0.2, rows=None):
    """alpha[k, h] of SDDMM -> LeakyReLU -> per-row softmax, float64 [nnz_sel, H]."""
    rp, cl = _c(rowptr, np.int32), _c(col, np.int32)
    sd, ss = _c(s_dst, np.float32), _c(s_src, np.float32)
    H = sd.shape[1]
    sel = _c(rows, np.int32)
    if sel is None:
        n_e = int(rp[-1])
    else:
        n_e = int(np.sum(rp[sel + 1].astype(np.int64) - rp[sel]))
    alpha = np.empty((n_e, H), dtype=np.float64)
    rc = _load().oracle_edge_softmax(rp.size - 1, ss.shape[0], int(rp[-1]), _p(rp), _p(cl), H,
                                     _p(sd), _p(ss), float(slope),
                                     0 if sel is None else sel.size, _p(sel), _p(alpha))
    _check(rc, "edge_softmax")
    return alpha


def gat(rowptr, col, s_dst, s_src, X, H, D, slope=0.2, alpha_in=None, x_dtype=None, rows=None):
    """Y[i,h,:] = sum_k alpha[k,h] X[col[k],h,:].  Returns (Y, Abs) float64 [n_sel, H*D]."""
    rp, cl = _c(rowptr, np.int32), _c(col, np.int32)
    sd, ss = _c(s_dst, np.float32), _c(s_src, np.float32)
    ai = _c(alpha_in, np.float32)
    X = np.ascontiguousarray(X)
    sel = _c(rows, np.int32)
    n_rows = rp.size - 1
    n_out = n_rows if sel is None else sel.size
    Y = np.empty((n_out, H * D), dtype=np.float64)
    A = np.empty((n_out, H * D), dtype=np.float64)
    rc = _load().oracle_gat(n_rows, X.shape[0], int(rp[-1]), _p(rp), _p(cl), H, D, _p(sd), _p(ss),
                            float(slope), _p(ai), _p(X), _x_code(X, x_dtype),
                            0 if sel is None else sel.size, _p(sel), _p(Y), _p(A))
    _check(rc, "gat")
    return Y, A


def _edges_of_rows(rp, sel):
    if sel is None:
        return int(rp[-1])
    return int(np.sum(rp[sel + 1].astype(np.int64) - rp[sel]))


def gat_backward(rowptr, col, s_dst, s_src, alpha, X, dY, H, D, slope=0.2, x_dtype=None,
                 dy_dtype=None, rows=None, cols=None, n_cols=None):
    """Gradients of the GAT layer (see oracle.c).  Returns a dict of float64 arrays:
    dalpha, dscore ([edges of the selected rows, H]), ds_dst ([rows, H]), ds_src
    ([cols, H]), dX ([cols, H*D]), each with its error scale under the key + "_abs"."""
    rp, cl = _c(rowptr, np.int32), _c(col, np.int32)
    sd, ss, al = _c(s_dst, np.float32), _c(s_src, np.float32), _c(alpha, np.float32)
    X, dY = np.ascontiguousarray(X), np.ascontiguousarray(dY)
    n_rows = rp.size - 1
    n_cols = X.shape[0] if n_cols is None else n_cols
    sel, csel = _c(rows, np.int32), _c(cols, np.int32)
    n_e = _edges_of_rows(rp, sel)
    n_r = n_rows if sel is None else sel.size
    n_c = n_cols if csel is None else csel.size
    out = {k: np.empty(shape, np.float64) for k, shape in (
        ("dalpha", (n_e, H)), ("dalpha_abs", (n_e, H)), ("dscore", (n_e, H)), ("dscore_abs", (n_e, H)),
        ("ds_dst", (n_r, H)), ("ds_dst_abs", (n_r, H)), ("ds_src", (n_c, H)), ("ds_src_abs", (n_c, H)),
        ("dX", (n_c, H * D)), ("dX_abs", (n_c, H * D)))}
    rc = _load().oracle_gat_backward(
        n_rows, n_cols, int(rp[-1]), _p(rp), _p(cl), H, D, _p(sd), _p(ss), float(slope), _p(al),
        _p(X), _x_code(X, x_dtype), _p(dY), _x_code(dY, dy_dtype),
        0 if sel is None else sel.size, _p(sel), _p(out["dalpha"]), _p(out["dalpha_abs"]),
        _p(out["dscore"]), _p(out["dscore_abs"]), _p(out["ds_dst"]), _p(out["ds_dst_abs"]),
        0 if csel is None else csel.size, _p(csel), _p(out["ds_src"]), _p(out["ds_src_abs"]),
        _p(out["dX"]), _p(out["dX_abs"]))
    _check(rc, "gat_backward")
    return out


def sddmm_dot(rowptr, col, P, Q, H, D, p_dtype=None, q_dtype=None, rows=None, n_cols=None):
    """out[k,h] = <P[i,h,:], Q[col[k],h,:]> (section 2.2 SDDMM per head).  Returns
    (out, Abs) float64 [edges of the selected rows, H]."""
    rp, cl = _c(rowptr, np.int32), _c(col, np.int32)
    P, Q = np.ascontiguousarray(P), np.ascontiguousarray(Q)
    n_rows = rp.size - 1
    n_cols = Q.shape[0] if n_cols is None else n_cols
    sel = _c(rows, np.int32)
    n_e = _edges_of_rows(rp, sel)
    out = np.empty((n_e, H), np.float64)
    ab = np.empty((n_e, H), np.float64)
    rc = _load().oracle_sddmm_dot(n_rows, n_cols, int(rp[-1]), _p(rp), _p(cl), H, D, _p(P),
                                  _x_code(P, p_dtype), _p(Q), _x_code(Q, q_dtype),
                                  0 if sel is None else sel.size, _p(sel), _p(out), _p(ab))
    _check(rc, "sddmm_dot")
    return out, ab


ACT = {"none": 0, "relu": 1, "elu": 2}


def epilogue(Y, bias=None, act="none"):
    """act(Y + bias) in place on a float64 [n, F] array (returns it)."""
    Y = np.ascontiguousarray(Y, dtype=np.float64)
    b = _c(bias, np.float32)
    n, F = Y.shape
    _check(_load().oracle_epilogue(n, F, _p(b), ACT[act], _p(Y)), "epilogue")
    return Y


def linear(X, W, bias=None, act="none", x_dtype=None, w_dtype=None):
    """Y = act(X W^T + bias) in float64 with its error scale.  X [n, k], W [m, k]
    (fp32 arrays, or uint16 bit patterns with explicit dtype codes)."""
    X, W = np.ascontiguousarray(X), np.ascontiguousarray(W)
    b = _c(bias, np.float32)
    n, k = X.shape
    m = W.shape[0]
    Y = np.empty((n, m), np.float64)
    A = np.empty((n, m), np.float64)
    _check(_load().oracle_linear(n, k, m, _p(X), _x_code(X, x_dtype), _p(W), _x_code(W, w_dtype),
                                 _p(b), ACT[act], _p(Y), _p(A)), "linear")
    return Y, A


def head_scores(Z, a_src, a_dst, H, D, z_dtype=None):
    """(s_src, s_dst, src_abs, dst_abs) float64 [n, H] for Z [n, H*D]."""
    Z = np.ascontiguousarray(Z)
    a_s, a_d = _c(a_src, np.float32), _c(a_dst, np.float32)
    n = Z.shape[0]
    out = [np.empty((n, H), np.float64) for _ in range(4)]
    _check(_load().oracle_head_scores(n, H, D, _p(Z), _x_code(Z, z_dtype), _p(a_s), _p(a_d),
                                      *[_p(o) for o in out]), "head_scores")
    return tuple(out)


def _row_max_over_edges(rowptr, col, per_row, per_col):
    """M[i, h] = max over the edges k of row i of per_row[i, h] + per_col[col[k], h] (0 when empty)."""
    rp = np.asarray(rowptr, np.int64)
    deg = np.diff(rp)
    rows = np.repeat(np.arange(rp.size - 1), deg)
    v = per_row[rows] + per_col[np.asarray(col)]
    M = np.zeros_like(per_row)
    nz = deg > 0
    if v.size:
        M[nz] = np.maximum.reduceat(v, rp[:-1][nz], axis=0)
    return M


def gcn_forward(rowptr, col, val, X, params, x_dtype=BF16, act_dtype=BF16, rows=None):
    """2-layer GCN inference with the activations stored in act_dtype between the
    steps, as the GPU pipeline stores them: Z1 = X W1^T, H1 = relu(A Z1 + b1),
    Z2 = H1 W2^T, Y = A Z2 + b2 (everything else in float64).
    Returns (Y, E): the output before its own rounding and an error scale E that
    bounds how far a one-unit difference in the rounding of any stored
    intermediate can move Y: each stage's scale is the stage applied to the
    absolute values of its inputs' scales (the activations are 1-Lipschitz).
    `rows` restricts the rows of the last aggregation."""
    W1, b1, W2, b2 = params["W1"], params["b1"], params["W2"], params["b2"]
    wd = params.get("w_dtype", BF16)
    aval = None if val is None else np.abs(np.asarray(val, np.float32))
    Z1, EZ1 = linear(X, W1, x_dtype=x_dtype, w_dtype=wd)
    H1, _ = spmm(rowptr, col, val, round_to(Z1, act_dtype), x_dtype=act_dtype)
    H1 = epilogue(H1, b1, "relu")
    EH1, _ = spmm(rowptr, col, aval, EZ1.astype(np.float32))
    EH1 += np.abs(np.asarray(b1, np.float64))[None, :]
    Z2, _ = linear(round_to(H1, act_dtype), W2, x_dtype=act_dtype, w_dtype=wd)
    EZ2, _ = linear(EH1.astype(np.float32), np.abs(decode(W2, wd)).astype(np.float32))
    Y, _ = spmm(rowptr, col, val, round_to(Z2, act_dtype), x_dtype=act_dtype, rows=rows)
    Y = epilogue(Y, b2, "none")
    EY, _ = spmm(rowptr, col, aval, EZ2.astype(np.float32), rows=rows)
    return Y, EY + np.abs(np.asarray(b2, np.float64))[None, :]


def _gat_layer(rowptr, col, Zs, EZ, a_src, a_dst, H, D, slope, bias, act, act_dtype, rows=None):
    """One GAT layer on stored features Zs [n, H*D] (act_dtype bits) with scale EZ:
    scores from the stored features, rounded to fp32 as they are stored; output and scale."""
    ss, sd, s_abs, d_abs = head_scores(Zs, a_src, a_dst, H, D, z_dtype=act_dtype)
    ss32, sd32 = ss.astype(np.float32), sd.astype(np.float32)
    Y, A = gat(rowptr, col, sd32, ss32, Zs, H, D, slope=slope, x_dtype=act_dtype, rows=rows)
    Y = epilogue(Y, bias, act)
    EY, _ = gat(rowptr, col, sd32, ss32, EZ.astype(np.float32), H, D, slope=slope, rows=rows)
    # a change of the scores by at most delta_e moves each weight by at most
    # 2 delta_e alpha; delta_e <= (scale of s_dst + scale of s_src) per edge
    M = _row_max_over_edges(rowptr, col, d_abs, s_abs)
    if rows is not None:
        M = M[np.asarray(rows)]
    EY += 2.0 * np.repeat(M, D, axis=1) * A
    if bias is not None:
        EY += np.abs(np.asarray(bias, np.float64))[None, :]
    return Y, EY


def gat_forward(rowptr, col, X, params, slope=0.2, x_dtype=BF16, act_dtype=BF16, rows=None):
    """2-layer GAT inference (layer 1: H heads of D concatenated, ELU; layer 2: one
    head of C outputs), activations stored in act_dtype, scores in fp32, the rest in
    float64.  Returns (Y, E) as gcn_forward."""
    H, D = np.asarray(params["a_src1"]).shape
    C = params["W2"].shape[0]
    wd = params.get("w_dtype", BF16)
    Z1, EZ1 = linear(X, params["W1"], x_dtype=x_dtype, w_dtype=wd)
    H1, EH1 = _gat_layer(rowptr, col, round_to(Z1, act_dtype), EZ1, params["a_src1"], params["a_dst1"],
                         H, D, slope, params["b1"], "elu", act_dtype)
    Z2, _ = linear(round_to(H1, act_dtype), params["W2"], x_dtype=act_dtype, w_dtype=wd)
    EZ2, _ = linear(EH1.astype(np.float32), np.abs(decode(params["W2"], wd)).astype(np.float32))
    return _gat_layer(rowptr, col, round_to(Z2, act_dtype), EZ2, params["a_src2"], params["a_dst2"],
                      1, C, slope, params["b2"], "none", act_dtype, rows=rows)


def philox4x32_10(counter, key):
    """The four 32-bit outputs of Philox4x32-10 for a 4-word counter and a 2-word key."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, np.uint32)
    _load().oracle_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def codec_layout(n, F, bits, group):
    """(groups per row, uint64 code words, fp32 stats) of a compressed n x F array."""
    ng = (F + group - 1) // group
    return ng, n * ng * (group // 64) * bits, n * ng * 2


def act_compress(A, bits, group, seed, a_dtype=None):
    """Codes (uint64 bit planes) and stats (fp32 min, step per group) of A [n, F]."""
    A = np.ascontiguousarray(A)
    n, F = A.shape
    _, n_words, n_stats = codec_layout(n, F, bits, group)
    codes = np.empty(n_words, np.uint64)
    stats = np.empty(n_stats, np.float32)
    _check(_load().oracle_act_compress(n, F, _p(A), _x_code(A, a_dtype), bits, group,
                                       ctypes.c_uint64(seed), _p(codes), _p(stats)), "act_compress")
    return codes, stats


def act_decompress(codes, stats, n, F, bits, group):
    out = np.empty((n, F), np.float32)
    _check(_load().oracle_act_decompress(n, F, bits, group, _p(np.ascontiguousarray(codes, np.uint64)),
                                         _p(np.ascontiguousarray(stats, np.float32)), _p(out)),
           "act_decompress")
    return out
