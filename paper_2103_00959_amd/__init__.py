"""MI355X-native GNN message-passing operators of the CogDL paper (arxiv 2103.00959, section 2.2).

Thin ctypes binding over ``libcogdl_mi355.so`` (see ``include/cogdl.h``):
argument marshalling only.  Every step runs in the library's HIP kernels on
the current torch stream; torch is used for device memory and streams.  The
binding fails loudly when the library or a GPU is missing: there is no CPU
fallback.

    spmm(rowptr, col, val, X, plan=None, out_dtype=None)          -> Y = A X
    gspmm(rowptr, col, val, X, reduce, compute=..., ...)          -> Eq. 1 with sum/mean/max, mul/add/sub/copy
    csr_to_csc(rowptr, col, val, n_cols)                          -> colptr, row_t, val_t, perm
    spmm_t(colptr, row_t, val_t, G, plan_t=None, out_dtype=None)  -> dX = A^T G
    sddmm_edge_softmax(rowptr, col, s_dst, s_src, slope, plan)    -> alpha [nnz, H]
    gat_aggregate(rowptr, col, s_dst, s_src, X, slope, ...)       -> Y [n, H, D] (, alpha)
    sddmm_dot(rowptr, col, P, Q)                                  -> <P[i,h], Q[j,h]> per edge
    gat_backward(rowptr, col, colptr, row_t, perm, ..., dY)       -> dX, dalpha, dscore, ds_dst, ds_src
    Plan(rowptr, nnz, max_feat, max_heads, mode, group_size)      -> the workload balancer
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcogdl_mi355.so")

COGDL_F32, COGDL_BF16, COGDL_F16 = 0, 1, 2
BALANCE = {"auto": 0, "row_split": 1, "neighbor_group": 2}
MODE_NAMES = {1: "row_split", 2: "neighbor_group"}
MAX_HEADS = 64
MAX_NNZ = 2**31 - 4097     # COGDL_MAX_NNZ: int32 edge ids with room for one batch past the end

_lib = None


class CogdlError(RuntimeError):
    pass


class _PlanInfo(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int32), ("nnz", ctypes.c_int64), ("group_size", ctypes.c_int32),
                ("max_feat", ctypes.c_int32), ("max_heads", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("n_units", ctypes.c_int32), ("n_long_units", ctypes.c_int32),
                ("n_split_rows", ctypes.c_int32),
                ("n_partials", ctypes.c_int32), ("device_bytes", ctypes.c_int64)]


def lib():
    """Load the HIP library (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (loads the HIP runtime the library binds to)
    if not os.path.exists(LIB_PATH):
        raise CogdlError(f"{LIB_PATH} is missing: build it with `python -m paper_2103_00959_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    L.cogdl_status_string.restype = ctypes.c_char_p
    L.cogdl_status_string.argtypes = [ctypes.c_int]
    L.cogdl_version.restype = i32
    L.cogdl_plan_create.argtypes = [i32, i64, P, i32, i32, ctypes.c_int, i32, P, ctypes.POINTER(P)]
    L.cogdl_plan_rebuild.argtypes = [P, P, P]
    L.cogdl_plan_create_sliced.argtypes = [i32, i64, P, P, i32, i32, i32, ctypes.c_int, i32, i32, P,
                                           ctypes.POINTER(P)]
    L.cogdl_plan_rebuild_sliced.argtypes = [P, P, P, P]
    L.cogdl_plan_destroy.argtypes = [P]
    L.cogdl_plan_query.argtypes = [P, P, ctypes.POINTER(_PlanInfo)]
    L.cogdl_plan_units.argtypes = [P, P, i64, P]
    L.cogdl_spmm.argtypes = [i32, i32, i64, P, P, P, i32, P, ctypes.c_int, P, ctypes.c_int, P, P]
    L.cogdl_gspmm.argtypes = [i32, i32, i64, P, P, P, i32, P, ctypes.c_int, P, ctypes.c_int,
                              ctypes.c_int, ctypes.c_int, P, ctypes.c_int, P, P, P]
    L.cogdl_gat_aggregate_act.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, f32, P, P,
                                          ctypes.c_int, P, ctypes.c_int, P, P, ctypes.c_int, P, P]
    L.cogdl_gat_aggregate_proj.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, f32, P, ctypes.c_int, P,
                                           ctypes.c_int, P, ctypes.c_int, P, P]
    L.cogdl_gat_aggregate_stats.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, P, f32, P, ctypes.c_int, P,
                                            ctypes.c_int, P, P, ctypes.c_int, P, P]
    L.cogdl_linear.argtypes = [i64, i32, i32, P, P, ctypes.c_int, P, ctypes.c_int, P, ctypes.c_int, P]
    L.cogdl_head_scores.argtypes = [i64, i32, i32, P, ctypes.c_int, P, P, P, P, P]
    L.cogdl_act_codec_size.argtypes = [i64, i32, i32, i32, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    L.cogdl_act_compress.argtypes = [i64, i32, P, ctypes.c_int, i32, i32, ctypes.c_uint64, P, P, P]
    L.cogdl_act_decompress.argtypes = [i64, i32, i32, i32, P, P, P, ctypes.c_int, P]
    L.cogdl_spmm_t.argtypes = [i32, i32, i64, P, P, P, i32, P, ctypes.c_int, P, ctypes.c_int, P, P]
    L.cogdl_csr_to_csc_workspace.argtypes = [i32, i32, i64, ctypes.POINTER(sz)]
    L.cogdl_csr_to_csc.argtypes = [i32, i32, i64, P, P, P, P, P, P, P, P, sz, P]
    L.cogdl_csr_to_csc_noalloc.argtypes = [i32, i32, i64, P, P, P, P, P, P, P, P]
    L.cogdl_sddmm_edge_softmax.argtypes = [i32, i32, i64, P, P, i32, P, P, f32, P, P, P]
    L.cogdl_gat_aggregate.argtypes = [i32, i32, i64, P, P, i32, i32, P, P, f32, P, P, ctypes.c_int,
                                      P, ctypes.c_int, P, P, P]
    L.cogdl_sddmm_dot.argtypes = [i32, i32, i64, P, P, i32, i32, P, ctypes.c_int, P, ctypes.c_int,
                                  P, P, P]
    L.cogdl_gat_backward.argtypes = [i32, i32, i64, P, P, P, P, P, i32, i32, P, P, f32, P, P,
                                     ctypes.c_int, P, ctypes.c_int, P, ctypes.c_int, P, P, P, P, P,
                                     P, P, P]
    L.cogdl_gat_backward_stats.argtypes = L.cogdl_gat_backward.argtypes
    L.cogdl_trace_enable.argtypes = [i32]
    L.cogdl_trace_filter.argtypes = [ctypes.c_char_p]
    L.cogdl_trace_count.restype = i32
    L.cogdl_trace_get.argtypes = [i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(f32)]
    for name in ("cogdl_trace_enable", "cogdl_trace_filter", "cogdl_trace_reset", "cogdl_trace_get", "cogdl_plan_create", "cogdl_plan_rebuild", "cogdl_plan_create_sliced", "cogdl_plan_rebuild_sliced", "cogdl_plan_destroy", "cogdl_plan_query",
                 "cogdl_plan_units", "cogdl_spmm", "cogdl_gspmm", "cogdl_spmm_t", "cogdl_csr_to_csc_workspace",
                 "cogdl_csr_to_csc", "cogdl_csr_to_csc_noalloc", "cogdl_sddmm_edge_softmax",
                 "cogdl_gat_aggregate",
                 "cogdl_sddmm_dot", "cogdl_gat_backward", "cogdl_gat_backward_stats",
                 "cogdl_gat_aggregate_act", "cogdl_gat_aggregate_proj", "cogdl_gat_aggregate_stats",
                 "cogdl_linear",
                 "cogdl_head_scores", "cogdl_act_codec_size", "cogdl_act_compress",
                 "cogdl_act_decompress"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int, what: str):
    if status != 0:
        msg = lib().cogdl_status_string(status).decode()
        raise CogdlError(f"{what}: {msg} (status {status})")


def _dtype_code(t) -> int:
    import torch
    codes = {torch.float32: COGDL_F32, torch.bfloat16: COGDL_BF16, torch.float16: COGDL_F16}
    if t.dtype not in codes:
        raise CogdlError(f"unsupported feature dtype {t.dtype}")
    return codes[t.dtype]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, name, dtype=None):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise CogdlError(f"{name} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise CogdlError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise CogdlError(f"{name} must be contiguous")
    return t


# Size checks.  The C ABI receives bare pointers and cannot see how large a
# tensor is, so every size the library will read or write through is checked
# here, before any device check and before anything is launched: a tensor of
# the wrong size would otherwise be read or written out of bounds on the GPU.
def _tensor(t, name):
    import torch
    if not isinstance(t, torch.Tensor):
        raise CogdlError(f"{name} must be a torch tensor, got {type(t).__name__}")
    return t


def _dims(t, name, ndim):
    _tensor(t, name)
    if t.dim() != ndim:
        raise CogdlError(f"{name} must have {ndim} dimensions, got shape {tuple(t.shape)}")
    return tuple(t.shape)


def _numel(t, name, n):
    """t is None, or a tensor of exactly n elements."""
    if t is None:
        return
    _tensor(t, name)
    if t.numel() != n:
        raise CogdlError(f"{name} has {t.numel()} elements, expected {n}")


def _at_least(t, name, n):
    if t is None:
        return
    _tensor(t, name)
    if t.numel() < n:
        raise CogdlError(f"{name} has {t.numel()} elements, needs at least {n}")


def _index_array(t, name):
    """A 1-D int32 index array (rowptr, col, ...): its element count."""
    _dims(t, name, 1)
    return t.numel()


def _rowptr_rows(rowptr, name="rowptr"):
    n = _index_array(rowptr, name)
    if n < 1:
        raise CogdlError(f"{name} needs at least one entry (n_rows + 1)")
    return n - 1


def _feat2(X, name):
    """(rows, width) of a feature matrix given as [rows, F] or [rows]."""
    _tensor(X, name)
    if X.dim() == 2:
        return X.shape[0], X.shape[1]
    if X.dim() == 1:
        return X.shape[0], 1
    raise CogdlError(f"{name} must be [rows, F] or [rows], got shape {tuple(X.shape)}")


def _plan_matches(plan, n_rows, nnz, name="plan"):
    if plan is not None and (plan.n_rows != n_rows or plan.nnz != nnz):
        raise CogdlError(f"{name} was built for {plan.n_rows} rows and {plan.nnz} nonzeros, "
                         f"the call has {n_rows} rows and {nnz} nonzeros")


class Plan:
    """The data-aware workload balancer (section 2.2): run once per graph."""

    def __init__(self, rowptr, nnz: int, max_feat: int, max_heads: int = 0, mode: str = "auto",
                 group_size: int = 0, col=None, n_cols: int | None = None, slice_min: int = 0):
        """With `col` (and `n_cols`), a column-sliced plan (cogdl_plan_create_sliced): long rows
        are also cut at 8 column-range boundaries and each range's units run on one XCD."""
        import torch
        self._h = None
        n_rows = _rowptr_rows(rowptr)
        if mode not in BALANCE:
            raise CogdlError(f"mode must be one of {sorted(BALANCE)}")
        self.sliced = col is not None
        if self.sliced:
            _index_array(col, "col")
            _numel(col, "col", int(nnz))
            if n_cols is None:
                raise CogdlError("a sliced plan needs n_cols")
        _dev(rowptr, "rowptr", torch.int32)
        self.rowptr = rowptr
        self.n_rows = n_rows
        self.nnz = int(nnz)
        h = ctypes.c_void_p()
        if self.sliced:
            _dev(col, "col", torch.int32)
            self.col = col
            _check(lib().cogdl_plan_create_sliced(self.n_rows, self.nnz, _ptr(rowptr), _ptr(col), int(n_cols),
                                                  int(max_feat), int(max_heads), BALANCE[mode], int(group_size),
                                                  int(slice_min), _stream(), ctypes.byref(h)),
                   "cogdl_plan_create_sliced")
        else:
            _check(lib().cogdl_plan_create(self.n_rows, self.nnz, _ptr(rowptr), int(max_feat),
                                           int(max_heads), BALANCE[mode], int(group_size), _stream(),
                                           ctypes.byref(h)), "cogdl_plan_create")
        self._h = h

    @property
    def handle(self):
        if self._h is None:
            raise CogdlError("plan destroyed")
        return self._h

    def rebuild(self, rowptr=None, col=None):
        import torch
        if rowptr is not None:
            _numel(rowptr, "rowptr", self.n_rows + 1)
            _index_array(rowptr, "rowptr")
        if col is not None:
            if not self.sliced:
                raise CogdlError("only a sliced plan is rebuilt with col")
            _numel(col, "col", self.nnz)
            _index_array(col, "col")
        if rowptr is not None:
            _dev(rowptr, "rowptr", torch.int32)
            self.rowptr = rowptr
        if self.sliced:
            if col is not None:
                _dev(col, "col", torch.int32)
                self.col = col
            _check(lib().cogdl_plan_rebuild_sliced(self.handle, _ptr(self.rowptr), _ptr(self.col), _stream()),
                   "cogdl_plan_rebuild_sliced")
        else:
            _check(lib().cogdl_plan_rebuild(self.handle, _ptr(self.rowptr), _stream()), "cogdl_plan_rebuild")

    def info(self) -> dict:
        inf = _PlanInfo()
        _check(lib().cogdl_plan_query(self.handle, _stream(), ctypes.byref(inf)), "cogdl_plan_query")
        d = {f: getattr(inf, f) for f, _ in _PlanInfo._fields_}
        d["mode_name"] = MODE_NAMES.get(d["mode"], "?")
        return d

    def units(self):
        import torch
        n = self.info()["n_units"]
        out = torch.empty((max(n, 1), 4), dtype=torch.int32, device="cuda")
        _check(lib().cogdl_plan_units(self.handle, _ptr(out), n, _stream()), "cogdl_plan_units")
        return out[:n]

    def close(self):
        if getattr(self, "_h", None) is not None:
            lib().cogdl_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def trace_enable(capacity: int = 4096):
    """Record HIP events around every library kernel launch (0 disables)."""
    _check(lib().cogdl_trace_enable(int(capacity)), "cogdl_trace_enable")


def trace_filter(names=None):
    """Record only the launches with these names (an iterable of str); None: all."""
    arg = None if names is None else ",".join(names).encode()
    _check(lib().cogdl_trace_filter(arg), "cogdl_trace_filter")


def trace_reset():
    _check(lib().cogdl_trace_reset(), "cogdl_trace_reset")


def trace_read() -> list:
    """[(kernel name, milliseconds)] of the launches recorded since the last reset."""
    L = lib()
    out = []
    for i in range(L.cogdl_trace_count()):
        name, ms = ctypes.c_char_p(), ctypes.c_float()
        _check(L.cogdl_trace_get(i, ctypes.byref(name), ctypes.byref(ms)), "cogdl_trace_get")
        out.append((name.value.decode(), ms.value))
    return out


def _plan_handle(plan):
    return None if plan is None else plan.handle


def _graph(rowptr, col, val=None, val_name="val"):
    """(n_rows, nnz) of a CSR (or CSC) graph, with the sizes of its arrays checked."""
    n_rows = _rowptr_rows(rowptr)
    nnz = _index_array(col, "col")
    _numel(val, val_name, nnz)
    return n_rows, nnz


def spmm(rowptr, col, val, X, plan: Plan | None = None, out_dtype=None, out=None):
    """Y[i] = sum_k val[k] * X[col[k]] over row i (Eq. 1, sum of products)."""
    import torch
    n_rows, nnz = _graph(rowptr, col, val)
    n_cols, F = _feat2(X, "X")
    _numel(out, "out", n_rows * F)
    _plan_matches(plan, n_rows, nnz)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32)
    _dev(val, "val", torch.float32), _dev(X, "X")
    if out is None:
        out = torch.empty((n_rows, F), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    _check(lib().cogdl_spmm(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), _ptr(val), F,
                            _ptr(X), _dtype_code(X), _ptr(out), _dtype_code(out), _plan_handle(plan),
                            _stream()), "cogdl_spmm")
    return out


REDUCE = {"sum": 0, "mean": 1, "max": 2}
COMPUTE = {"mul": 0, "add": 1, "sub": 2, "copy": 3}
ACT = {"none": 0, "relu": 1, "elu": 2}


def gspmm(rowptr, col, val, X, reduce: str = "sum", plan: Plan | None = None, out_dtype=None,
          out=None, return_arg: bool = False, arg=None, compute: str = "mul", bias=None,
          act: str = "none"):
    """Eq. 1 with reduce = sum, mean or max over the edges k of row i of the
    message val[k] * x (compute "mul"), x + val[k] ("add"), x - val[k] ("sub")
    or x ("copy"), x = X[col[k]]; then act(. + bias) (bias fp32 [F] or None).

    For max, ``return_arg`` also returns the int32 edge id of the first edge
    attaining each output (-1 on empty rows); max keeps X's dtype or fp32."""
    import torch
    if reduce not in REDUCE:
        raise ValueError(f"reduce must be one of {sorted(REDUCE)}")
    if compute not in COMPUTE:
        raise ValueError(f"compute must be one of {sorted(COMPUTE)}")
    if act not in ACT:
        raise ValueError(f"act must be one of {sorted(ACT)}")
    if (return_arg or arg is not None) and reduce != "max":
        raise ValueError("return_arg / arg need reduce='max'")
    n_rows, nnz = _graph(rowptr, col, val)
    n_cols, F = _feat2(X, "X")
    _numel(out, "out", n_rows * F)
    _numel(arg, "arg", n_rows * F)
    _numel(bias, "bias", F)
    _plan_matches(plan, n_rows, nnz)
    _dev(bias, "bias", torch.float32)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32)
    _dev(val, "val", torch.float32), _dev(X, "X")
    if out is None:
        out = torch.empty((n_rows, F), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    if return_arg and arg is None:
        arg = torch.empty((n_rows, F), dtype=torch.int32, device=X.device)
    _dev(arg, "arg", torch.int32)
    _check(lib().cogdl_gspmm(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), _ptr(val), F,
                             _ptr(X), _dtype_code(X), _ptr(out), _dtype_code(out), REDUCE[reduce],
                             COMPUTE[compute], _ptr(bias), ACT[act], _ptr(arg), _plan_handle(plan),
                             _stream()), "cogdl_gspmm")
    return (out, arg) if return_arg else out


def csr_to_csc_workspace(n_rows: int, n_cols: int, nnz: int) -> int:
    b = ctypes.c_size_t()
    _check(lib().cogdl_csr_to_csc_workspace(n_rows, n_cols, nnz, ctypes.byref(b)),
           "cogdl_csr_to_csc_workspace")
    return b.value


def csr_to_csc(rowptr, col, val, n_cols: int, workspace=None, with_perm: bool = True):
    """Stable transpose: (colptr, row_t, val_t, perm); inside a column edges keep CSR order."""
    import torch
    n_rows, nnz = _graph(rowptr, col, val)
    n_cols = int(n_cols)
    if n_cols < 0:
        raise CogdlError("n_cols must be >= 0")
    if workspace is not None:
        _dims(workspace, "workspace", 1)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(val, "val", torch.float32)
    dev = rowptr.device
    colptr = torch.empty(n_cols + 1, dtype=torch.int32, device=dev)
    row_t = torch.empty(nnz, dtype=torch.int32, device=dev)
    val_t = None if val is None else torch.empty(nnz, dtype=torch.float32, device=dev)
    perm = torch.empty(nnz, dtype=torch.int32, device=dev) if with_perm else None
    need = csr_to_csc_workspace(n_rows, n_cols, nnz)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    _dev(workspace, "workspace")
    _check(lib().cogdl_csr_to_csc(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), _ptr(val),
                                  _ptr(colptr), _ptr(row_t), _ptr(val_t), _ptr(perm), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream()),
           "cogdl_csr_to_csc")
    return colptr, row_t, val_t, perm


def csr_to_csc_noalloc(rowptr, col, val, n_cols: int, out=None, with_perm: bool = True):
    """The transpose of csr_to_csc through cogdl_csr_to_csc_noalloc, which allocates nothing
    (its scratch is the library's static per-GPU array, so graphs up to about 1.6M edges).
    ``out`` may supply (colptr, row_t, val_t, perm); calls on one GPU must not overlap."""
    import torch
    n_rows, nnz = _graph(rowptr, col, val)
    n_cols = int(n_cols)
    if n_cols < 0:
        raise CogdlError("n_cols must be >= 0")
    if out is not None:
        colptr, row_t, val_t, perm = out
        _numel(colptr, "colptr", n_cols + 1)
        _numel(row_t, "row_t", nnz)
        _numel(val_t, "val_t", nnz)
        _numel(perm, "perm", nnz)
    need, limit = csr_to_csc_workspace(n_rows, n_cols, nnz), 64 << 20   # COGDL_NOALLOC_SCRATCH_BYTES
    if need > limit:
        raise CogdlError(f"cogdl_csr_to_csc_noalloc: a graph of {nnz} edges needs {need} bytes of "
                         f"scratch, the static scratch holds {limit}: use csr_to_csc with a workspace")
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(val, "val", torch.float32)
    if out is None:
        dev = rowptr.device
        colptr = torch.empty(n_cols + 1, dtype=torch.int32, device=dev)
        row_t = torch.empty(nnz, dtype=torch.int32, device=dev)
        val_t = None if val is None else torch.empty(nnz, dtype=torch.float32, device=dev)
        perm = torch.empty(nnz, dtype=torch.int32, device=dev) if with_perm else None
    for t, name, dt in ((colptr, "colptr", torch.int32), (row_t, "row_t", torch.int32),
                        (val_t, "val_t", torch.float32), (perm, "perm", torch.int32)):
        _dev(t, name, dt)
    _check(lib().cogdl_csr_to_csc_noalloc(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), _ptr(val),
                                          _ptr(colptr), _ptr(row_t), _ptr(val_t), _ptr(perm),
                                          _stream()), "cogdl_csr_to_csc_noalloc")
    return colptr, row_t, val_t, perm


def spmm_t(colptr, row_t, val_t, G, plan_t: Plan | None = None, out_dtype=None, out=None):
    """dX = A^T G from the CSC arrays of A; G is n_rows x F."""
    import torch
    n_cols = _rowptr_rows(colptr, "colptr")
    nnz = _index_array(row_t, "row_t")
    _numel(val_t, "val_t", nnz)
    n_rows, F = _feat2(G, "G")
    _numel(out, "out", n_cols * F)
    _plan_matches(plan_t, n_cols, nnz, "plan_t")
    _dev(colptr, "colptr", torch.int32), _dev(row_t, "row_t", torch.int32)
    _dev(val_t, "val_t", torch.float32), _dev(G, "G")
    if out is None:
        out = torch.empty((n_cols, F), dtype=out_dtype or G.dtype, device=G.device)
    _dev(out, "out")
    _check(lib().cogdl_spmm_t(n_rows, n_cols, nnz, _ptr(colptr), _ptr(row_t),
                              _ptr(val_t), F, _ptr(G), _dtype_code(G), _ptr(out), _dtype_code(out),
                              _plan_handle(plan_t), _stream()), "cogdl_spmm_t")
    return out


def _scores(t, name, rows, H):
    """A per-node score array [rows, H] (fp32)."""
    shape = _dims(t, name, 2)
    if shape != (rows, H):
        raise CogdlError(f"{name} must be [{rows}, {H}], got {shape}")


def sddmm_edge_softmax(rowptr, col, s_dst, s_src, negative_slope: float = 0.2,
                       plan: Plan | None = None, out=None):
    """alpha[k, h] = softmax over row i of LeakyReLU(s_dst[i, h] + s_src[col[k], h])."""
    import torch
    n_rows, nnz = _graph(rowptr, col)
    _dims(s_src, "s_src", 2)
    n_cols, H = s_src.shape
    _scores(s_dst, "s_dst", n_rows, H)
    _numel(out, "alpha", nnz * H)
    _plan_matches(plan, n_rows, nnz)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32)
    _dev(s_dst, "s_dst", torch.float32), _dev(s_src, "s_src", torch.float32)
    if out is None:
        out = torch.empty((nnz, H), dtype=torch.float32, device=col.device)
    _dev(out, "alpha", torch.float32)
    _check(lib().cogdl_sddmm_edge_softmax(n_rows, n_cols, nnz, _ptr(rowptr),
                                          _ptr(col), H, _ptr(s_dst), _ptr(s_src),
                                          float(negative_slope), _ptr(out), _plan_handle(plan),
                                          _stream()), "cogdl_sddmm_edge_softmax")
    return out


def gat_aggregate(rowptr, col, s_dst, s_src, X, negative_slope: float = 0.2, alpha_in=None,
                  return_alpha: bool = False, plan: Plan | None = None, out_dtype=None, out=None,
                  alpha_out=None, bias=None, act: str = "none"):
    """Fused GAT aggregation.  X is [n_cols, H, D]; returns Y [n_rows, H, D] (and alpha).
    With bias (fp32 [H*D]) or act, Y = act(aggregate + bias) (cogdl_gat_aggregate_act)."""
    import torch
    if act not in ACT:
        raise ValueError(f"act must be one of {sorted(ACT)}")
    n_rows, nnz = _graph(rowptr, col)
    n_cols, H, D = _dims(X, "X", 3)
    if alpha_in is None:
        _scores(s_dst, "s_dst", n_rows, H)
        _scores(s_src, "s_src", n_cols, H)
    else:
        if s_dst is not None:
            _scores(s_dst, "s_dst", n_rows, H)
        if s_src is not None:
            _scores(s_src, "s_src", n_cols, H)
        _numel(alpha_in, "alpha_in", nnz * H)
    _numel(out, "out", n_rows * H * D)
    _numel(alpha_out, "alpha_out", nnz * H)
    _numel(bias, "bias", H * D)
    _plan_matches(plan, n_rows, nnz)
    _dev(bias, "bias", torch.float32)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(X, "X")
    _dev(s_dst, "s_dst", torch.float32), _dev(s_src, "s_src", torch.float32)
    _dev(alpha_in, "alpha_in", torch.float32)
    if out is None:
        out = torch.empty((n_rows, H, D), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    if return_alpha and alpha_out is None:
        alpha_out = torch.empty((nnz, H), dtype=torch.float32, device=X.device)
    _dev(alpha_out, "alpha_out", torch.float32)
    if bias is None and act == "none":
        _check(lib().cogdl_gat_aggregate(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), H, D,
                                         _ptr(s_dst), _ptr(s_src), float(negative_slope),
                                         _ptr(alpha_in), _ptr(X), _dtype_code(X), _ptr(out),
                                         _dtype_code(out), _ptr(alpha_out), _plan_handle(plan),
                                         _stream()), "cogdl_gat_aggregate")
    else:
        _check(lib().cogdl_gat_aggregate_act(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), H, D,
                                             _ptr(s_dst), _ptr(s_src), float(negative_slope),
                                             _ptr(alpha_in), _ptr(X), _dtype_code(X), _ptr(out),
                                             _dtype_code(out), _ptr(alpha_out), _ptr(bias), ACT[act],
                                             _plan_handle(plan), _stream()), "cogdl_gat_aggregate_act")
    return (out, alpha_out) if return_alpha else out


def gat_aggregate_proj(rowptr, col, s_dst, a_src, X, negative_slope: float = 0.2,
                       plan: Plan | None = None, out_dtype=None, out=None, bias=None, act: str = "none"):
    """Fused GAT aggregation with the source scores projected from the gathered rows:
    s_src[j, h] = <X[j, h, :], a_src[h, :]> inside the kernel (cogdl_gat_aggregate_proj).
    X [n_cols, H, D] with D * itemsize a multiple of 16 bytes; a_src fp32 [H, D]."""
    import torch
    if act not in ACT:
        raise ValueError(f"act must be one of {sorted(ACT)}")
    n_rows, nnz = _graph(rowptr, col)
    n_cols, H, D = _dims(X, "X", 3)
    _scores(s_dst, "s_dst", n_rows, H)
    _numel(a_src, "a_src", H * D)
    _numel(out, "out", n_rows * H * D)
    _numel(bias, "bias", H * D)
    _plan_matches(plan, n_rows, nnz)
    _dev(bias, "bias", torch.float32), _dev(a_src, "a_src", torch.float32)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(X, "X")
    _dev(s_dst, "s_dst", torch.float32)
    if out is None:
        out = torch.empty((n_rows, H, D), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    _check(lib().cogdl_gat_aggregate_proj(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), H, D, _ptr(s_dst),
                                          _ptr(a_src), float(negative_slope), _ptr(X), _dtype_code(X),
                                          _ptr(out), _dtype_code(out), _ptr(bias), ACT[act],
                                          _plan_handle(plan), _stream()), "cogdl_gat_aggregate_proj")
    return out


def gat_aggregate_stats(rowptr, col, s_dst, X, s_src=None, a_src=None, negative_slope: float = 0.2,
                        plan: Plan | None = None, out_dtype=None, out=None, stats_out=None, bias=None,
                        act: str = "none"):
    """The GAT aggregation of a training step: returns (Y, row_stats), row_stats fp32
    [n_rows, 2, H] = the final (max score, 1 / normalizer) of each row's softmax per head, from
    which gat_backward(row_stats=...) rebuilds every weight instead of reading alpha.  Exactly
    one of s_src (scores given) and a_src (projected from X, as gat_aggregate_proj)."""
    import torch
    if act not in ACT:
        raise ValueError(f"act must be one of {sorted(ACT)}")
    if (s_src is None) == (a_src is None):
        raise CogdlError("give exactly one of s_src and a_src")
    n_rows, nnz = _graph(rowptr, col)
    n_cols, H, D = _dims(X, "X", 3)
    _scores(s_dst, "s_dst", n_rows, H)
    if s_src is not None:
        _scores(s_src, "s_src", n_cols, H)
    else:
        _numel(a_src, "a_src", H * D)
    _numel(out, "out", n_rows * H * D)
    _numel(stats_out, "stats_out", n_rows * 2 * H)
    _numel(bias, "bias", H * D)
    _plan_matches(plan, n_rows, nnz)
    _dev(bias, "bias", torch.float32), _dev(a_src, "a_src", torch.float32)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(X, "X")
    _dev(s_dst, "s_dst", torch.float32), _dev(s_src, "s_src", torch.float32)
    if out is None:
        out = torch.empty((n_rows, H, D), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    if stats_out is None:
        stats_out = torch.empty((n_rows, 2, H), dtype=torch.float32, device=X.device)
    _dev(stats_out, "stats_out", torch.float32)
    _check(lib().cogdl_gat_aggregate_stats(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), H, D, _ptr(s_dst),
                                           _ptr(s_src), _ptr(a_src), float(negative_slope), _ptr(X),
                                           _dtype_code(X), _ptr(out), _dtype_code(out), _ptr(stats_out),
                                           _ptr(bias), ACT[act], _plan_handle(plan), _stream()),
           "cogdl_gat_aggregate_stats")
    return out, stats_out


def sddmm_dot(rowptr, col, P, Q, plan: Plan | None = None, out=None):
    """out[k, h] = <P[i, h, :], Q[col[k], h, :]> for every edge k = (i, col[k]):
    the SDDMM of section 2.2 per head.  P is [n_rows, H, D], Q [n_cols, H, D]."""
    import torch
    n_rows, nnz = _graph(rowptr, col)
    pr, H, D = _dims(P, "P", 3)
    n_cols, qh, qd = _dims(Q, "Q", 3)
    if (qh, qd) != (H, D):
        raise CogdlError("P and Q must be [n, H, D] with the same H and D")
    if pr != n_rows:
        raise CogdlError(f"P has {pr} rows, the graph {n_rows}")
    _numel(out, "out", nnz * H)
    _plan_matches(plan, n_rows, nnz)
    _dev(rowptr, "rowptr", torch.int32), _dev(col, "col", torch.int32), _dev(P, "P"), _dev(Q, "Q")
    if out is None:
        out = torch.empty((nnz, H), dtype=torch.float32, device=P.device)
    _dev(out, "out", torch.float32)
    _check(lib().cogdl_sddmm_dot(n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), H, D, _ptr(P),
                                 _dtype_code(P), _ptr(Q), _dtype_code(Q), _ptr(out), _plan_handle(plan),
                                 _stream()), "cogdl_sddmm_dot")
    return out


def gat_backward(rowptr, col, colptr, row_t, perm, s_dst, s_src, alpha, X, dY,
                 negative_slope: float = 0.2, plan: Plan | None = None, plan_t: Plan | None = None,
                 dx_dtype=None, out=None, row_stats=None):
    """Gradients of gat_aggregate for dY = dL/dY.  X is [n_cols, H, D], dY [n_rows, H, D],
    alpha [nnz, H] the forward weights; (colptr, row_t, perm) the CSC from csr_to_csc.
    Returns dict(dX, dalpha, dscore, ds_dst, ds_src, edge_work); ``out`` may supply these
    tensors, and ``out={"dalpha": None, "dscore": None}`` (either or both) leaves those
    outputs out.  edge_work (fp32, 2 nnz H) is the library's scratch between its two passes:
    it ends holding the pair (alpha, dscore) of every edge and head.  With alpha None and
    row_stats (from gat_aggregate_stats) the weights are rebuilt instead of read
    (cogdl_gat_backward_stats)."""
    import torch
    n_rows, nnz = _graph(rowptr, col)
    n_cols, H, D = _dims(X, "X", 3)
    if _dims(dY, "dY", 3) != (n_rows, H, D):
        raise CogdlError(f"dY must be [{n_rows}, {H}, {D}], got {tuple(dY.shape)}")
    _numel(colptr, "colptr", n_cols + 1)
    _index_array(colptr, "colptr")
    for t, name in ((row_t, "row_t"), (perm, "perm")):
        _numel(t, name, nnz)
        _index_array(t, name)
    _scores(s_dst, "s_dst", n_rows, H)
    _scores(s_src, "s_src", n_cols, H)
    if (alpha is None) == (row_stats is None):
        raise CogdlError("give exactly one of alpha and row_stats")
    _numel(alpha, "alpha", nnz * H)
    _numel(row_stats, "row_stats", n_rows * 2 * H)
    o = dict(out or {})
    sizes = {"dX": n_cols * H * D, "dalpha": nnz * H, "dscore": nnz * H, "ds_dst": n_rows * H,
             "ds_src": n_cols * H, "edge_work": 2 * nnz * H}
    for k in o:
        if k not in sizes:
            raise CogdlError(f"unknown output {k!r}")
        if o[k] is None and k not in ("dalpha", "dscore"):
            raise CogdlError(f"output {k!r} is required")
        if o[k] is not None:
            _numel(o[k], k, sizes[k])
    _plan_matches(plan, n_rows, nnz)
    _plan_matches(plan_t, n_cols, nnz, "plan_t")
    for t, name, dt in ((rowptr, "rowptr", torch.int32), (col, "col", torch.int32),
                        (colptr, "colptr", torch.int32), (row_t, "row_t", torch.int32),
                        (perm, "perm", torch.int32), (s_dst, "s_dst", torch.float32),
                        (s_src, "s_src", torch.float32), (alpha, "alpha", torch.float32),
                        (row_stats, "row_stats", torch.float32)):
        _dev(t, name, dt)
    _dev(X, "X"), _dev(dY, "dY")
    dev = X.device
    o.setdefault("dX", torch.empty((n_cols, H, D), dtype=dx_dtype or X.dtype, device=dev))
    o.setdefault("dalpha", torch.empty((nnz, H), dtype=torch.float32, device=dev))
    o.setdefault("dscore", torch.empty((nnz, H), dtype=torch.float32, device=dev))
    o.setdefault("ds_dst", torch.empty((n_rows, H), dtype=torch.float32, device=dev))
    o.setdefault("ds_src", torch.empty((n_cols, H), dtype=torch.float32, device=dev))
    o.setdefault("edge_work", torch.empty((nnz, H, 2), dtype=torch.float32, device=dev))
    _dev(o["dX"], "dX")
    for k in ("dalpha", "dscore", "ds_dst", "ds_src", "edge_work"):
        if o[k] is not None:
            _dev(o[k], k, torch.float32)
    fn = "cogdl_gat_backward" if row_stats is None else "cogdl_gat_backward_stats"
    _check(getattr(lib(), fn)(
        n_rows, n_cols, nnz, _ptr(rowptr), _ptr(col), _ptr(colptr), _ptr(row_t), _ptr(perm), H, D,
        _ptr(s_dst), _ptr(s_src), float(negative_slope), _ptr(alpha if row_stats is None else row_stats),
        _ptr(X), _dtype_code(X), _ptr(dY), _dtype_code(dY), _ptr(o["dX"]), _dtype_code(o["dX"]),
        _ptr(o["dalpha"]), _ptr(o["dscore"]), _ptr(o["ds_dst"]), _ptr(o["ds_src"]), _ptr(o["edge_work"]),
        _plan_handle(plan), _plan_handle(plan_t), _stream()), fn)
    return o


def linear(X, W, bias=None, act: str = "none", out_dtype=None, out=None):
    """Y = act(X W^T + bias) on the matrix cores.  X [n, k] and W [m, k] (a layer's out x in
    weights) both bf16 or both fp16; bias fp32 [m] or None."""
    import torch
    if act not in ACT:
        raise ValueError(f"act must be one of {sorted(ACT)}")
    n, k = _dims(X, "X", 2)
    m, kw = _dims(W, "W", 2)
    if kw != k or X.dtype != W.dtype:
        raise CogdlError("X must be [n, k] and W [m, k] of the same dtype")
    _numel(bias, "bias", m)
    _numel(out, "out", n * m)
    _dev(X, "X"), _dev(W, "W"), _dev(bias, "bias", torch.float32)
    if out is None:
        out = torch.empty((n, m), dtype=out_dtype or X.dtype, device=X.device)
    _dev(out, "out")
    _check(lib().cogdl_linear(n, k, m, _ptr(X), _ptr(W), _dtype_code(X), _ptr(bias), ACT[act],
                              _ptr(out), _dtype_code(out), _stream()), "cogdl_linear")
    return out


def head_scores(Z, a_src, a_dst):
    """s_src[i, h] = <Z[i, h, :], a_src[h]>, s_dst likewise; Z [n, H, D], a_* fp32 [H, D].
    Either vector may be None; its scores are then not computed (returned as None)."""
    import torch
    n, H, D = _dims(Z, "Z", 3)
    if a_src is None and a_dst is None:
        raise CogdlError("head_scores needs a_src or a_dst")
    _numel(a_src, "a_src", H * D)
    _numel(a_dst, "a_dst", H * D)
    _dev(Z, "Z"), _dev(a_src, "a_src", torch.float32), _dev(a_dst, "a_dst", torch.float32)
    s_src = None if a_src is None else torch.empty((n, H), dtype=torch.float32, device=Z.device)
    s_dst = None if a_dst is None else torch.empty((n, H), dtype=torch.float32, device=Z.device)
    _check(lib().cogdl_head_scores(n, H, D, _ptr(Z), _dtype_code(Z), _ptr(a_src), _ptr(a_dst),
                                   _ptr(s_src), _ptr(s_dst), _stream()), "cogdl_head_scores")
    return s_src, s_dst


def _padded_output_layer(params, names_rows, names_cols):
    """The output layer's parameters with the output count padded to a multiple of 8 (zero
    rows / entries), prepared once per parameter dict: the aggregation then gathers
    16-byte vectors instead of single 16-bit elements of rows like 41 classes wide.  The
    padded outputs are exactly zero and are sliced away."""
    import torch
    key = "_padded_output_layer"
    if key not in params:
        C = params[names_rows[0]].shape[0]
        C8 = (C + 7) // 8 * 8
        pad = {}
        for n_ in names_rows:                     # [C, ...] -> [C8, ...]
            t = params[n_]
            z = torch.zeros((C8,) + tuple(t.shape[1:]), dtype=t.dtype, device=t.device)
            z[:C] = t
            pad[n_] = z
        for n_ in names_cols:                     # [1, C] -> [1, C8]
            t = params[n_]
            z = torch.zeros((t.shape[0], C8), dtype=t.dtype, device=t.device)
            z[:, :C] = t
            pad[n_] = z
        params[key] = (C, C8, pad)
    return params[key]


def gcn_forward(rowptr, col, val, X, params, plan: Plan | None = None):
    """2-layer GCN inference: H1 = relu(A (X W1^T) + b1), Y = A (H1 W2^T) + b2, every step a
    library kernel (dense layers on the matrix cores, aggregations with the bias and
    activation in their epilogue).  params: dict of W1 [hid, in], b1 [hid], W2 [out, hid],
    b2 [out]; activations stay in X's dtype.  Returns Y [n, out] (a view of the padded
    output when out is not a multiple of 8)."""
    C, C8, pad = _padded_output_layer(params, ("W2", "b2"), ())
    Z1 = linear(X, params["W1"])
    H1 = gspmm(rowptr, col, val, Z1, "sum", plan=plan, bias=params["b1"], act="relu")
    Z2 = linear(H1, pad["W2"])
    Y = gspmm(rowptr, col, val, Z2, "sum", plan=plan, bias=pad["b2"], act="none")
    return Y if C8 == C else Y[:, :C]


def _proj_ok(Z):
    """Whether cogdl_gat_aggregate_proj takes heads of this shape: [n, H, D] with each head a
    power-of-two number of 16-byte vectors."""
    per = 16 // Z.element_size()
    D = Z.shape[2]
    return D % per == 0 and ((D // per) & (D // per - 1)) == 0 and Z.data_ptr() % 16 == 0


def gat_forward(rowptr, col, X, params, negative_slope: float = 0.2, plan: Plan | None = None):
    """2-layer GAT inference: layer 1 with H heads of D (concatenated, ELU), layer 2 with one
    head of C outputs.  params: W1 [H*D, in], a_src1 / a_dst1 [H, D], b1 [H*D], W2 [C, H*D],
    a_src2 / a_dst2 [1, C], b2 [C].  Returns Y [n, C] (a view of the padded output when C is
    not a multiple of 8)."""
    H, D = params["a_src1"].shape
    C, C8, pad = _padded_output_layer(params, ("W2", "b2"), ("a_src2", "a_dst2"))
    n = X.shape[0]
    Z1 = linear(X, params["W1"]).view(n, H, D)
    if _proj_ok(Z1):
        # source scores formed from the rows the aggregation gathers: only s_dst is precomputed
        _, s_dst = head_scores(Z1, None, params["a_dst1"])
        H1 = gat_aggregate_proj(rowptr, col, s_dst, params["a_src1"], Z1, negative_slope, plan=plan,
                                bias=params["b1"], act="elu")
    else:
        s_src, s_dst = head_scores(Z1, params["a_src1"], params["a_dst1"])
        H1 = gat_aggregate(rowptr, col, s_dst, s_src, Z1, negative_slope, plan=plan, bias=params["b1"],
                           act="elu")
    Z2 = linear(H1.view(n, H * D), pad["W2"]).view(n, 1, C8)
    s_src2, s_dst2 = head_scores(Z2, pad["a_src2"], pad["a_dst2"])
    Y = gat_aggregate(rowptr, col, s_dst2, s_src2, Z2, negative_slope, plan=plan,
                      bias=pad["b2"]).view(n, C8)
    return Y if C8 == C else Y[:, :C]


def act_codec_size(n: int, F: int, bits: int, group: int):
    """(uint64 code words, fp32 stats) of a compressed n x F activation array."""
    w, st = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().cogdl_act_codec_size(n, F, bits, group, ctypes.byref(w), ctypes.byref(st)),
           "cogdl_act_codec_size")
    return w.value, st.value


def act_compress(A, bits: int, group: int, seed: int, codes=None, stats=None):
    """Per-group `bits`-bit stochastic quantization of A [n, F]: returns (codes int64 view of
    the uint64 bit planes, stats fp32 [groups, 2] = (min, step))."""
    import torch
    n, F = _dims(A, "A", 2)
    words, nst = act_codec_size(n, F, bits, group)
    _at_least(codes, "codes", words)
    _at_least(stats, "stats", nst)
    _dev(A, "A")
    if codes is None:
        codes = torch.empty(max(words, 1), dtype=torch.int64, device=A.device)
    if stats is None:
        stats = torch.empty(max(nst, 1), dtype=torch.float32, device=A.device)
    _dev(codes, "codes", torch.int64), _dev(stats, "stats", torch.float32)
    _check(lib().cogdl_act_compress(n, F, _ptr(A), _dtype_code(A), bits, group,
                                    ctypes.c_uint64(seed & 0xFFFFFFFFFFFFFFFF), _ptr(codes),
                                    _ptr(stats), _stream()), "cogdl_act_compress")
    return codes[:words], stats[:nst]


def act_decompress(codes, stats, n: int, F: int, bits: int, group: int, out_dtype=None, out=None):
    import torch
    words, nst = act_codec_size(n, F, bits, group)
    _at_least(codes, "codes", words)
    _at_least(stats, "stats", nst)
    _numel(out, "out", n * F)
    _dev(codes, "codes", torch.int64), _dev(stats, "stats", torch.float32)
    if out is None:
        out = torch.empty((n, F), dtype=out_dtype or torch.float32, device=codes.device)
    _dev(out, "out")
    _check(lib().cogdl_act_decompress(n, F, bits, group, _ptr(codes), _ptr(stats), _ptr(out),
                                      _dtype_code(out), _stream()), "cogdl_act_decompress")
    return out
