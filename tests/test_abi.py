"""C-ABI contract tests that need no GPU: the library loads, exports every
entry point the header declares, and rejects bad arguments on the host before
anything is launched (only calls whose validation fails are made here)."""
import ctypes
import os
import re

import pytest

import paper_2103_00959_amd as cg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cogdl.h")

OK, INVALID, DTYPE, PLAN, NOMEM, LAUNCH, TOO_LARGE = range(7)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(cg.LIB_PATH):
        from paper_2103_00959_amd import build
        build.build(verbose=False)
    return cg.lib()


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cogdl_[a-z_0-9]+)\s*\(", text)))


def test_header_symbols_exported(L):
    syms = declared_symbols()
    assert len(syms) >= 13
    for s in syms:
        assert hasattr(L, s), s


def test_calibration_library_exports_and_validation():
    """libcogdl_calib.so (counter calibration kernels) exports what include/cogdl_calib.h
    declares and refuses bad arguments on the host (nothing is launched here)."""
    from paper_2103_00959_amd import build
    if not os.path.exists(build.CALIB_LIB):
        build.build(verbose=False)
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "cogdl_calib.h")).read(), flags=re.S)
    syms = sorted(set(re.findall(r"\b(cogdl_calib_[a-z_0-9]+)\s*\(", text)))
    assert syms == ["cogdl_calib_copy", "cogdl_calib_gather", "cogdl_calib_read"]
    import bench
    C = bench.calib_lib()
    for s_ in syms:
        assert hasattr(C, s_)
    A = _p(0x100000)                       # 128-byte aligned, never dereferenced
    assert C.cogdl_calib_read(A, 100, A, None) == 1             # not a multiple of 16
    assert C.cogdl_calib_read(_p(0x100008), 160, A, None) == 1  # misaligned
    assert C.cogdl_calib_read(None, 160, A, None) == 1
    assert C.cogdl_calib_copy(A, A, 0, None) == 1
    assert C.cogdl_calib_copy(A, _p(0x100004), 160, None) == 1
    assert C.cogdl_calib_gather(A, 128, 48, A, 10, A, None) == 1    # row size
    assert C.cogdl_calib_gather(A, 64, 16, A, 10, A, None) == 1     # stride not a line multiple
    assert C.cogdl_calib_gather(_p(0x100040), 128, 16, A, 10, A, None) == 1
    assert C.cogdl_calib_gather(A, 128, 16, A, 0, A, None) == 1


def test_status_strings_and_version(L):
    for code in range(7):
        assert len(L.cogdl_status_string(code)) > 0
    assert L.cogdl_status_string(99) == b"unknown status"
    assert L.cogdl_version() >= 100


def _max_nnz():
    m = re.search(r"#define COGDL_MAX_NNZ (\d+)LL", open(HEADER).read())
    return int(m.group(1))


def test_max_nnz_limit(L):
    """Edge counts above COGDL_MAX_NNZ (2^31 - 4097) are refused by every entry point that
    takes one: int32 edge ids need room for a batch of indices past the last edge."""
    import paper_2103_00959_amd as cgm
    big = _max_nnz() + 1
    assert big == (1 << 31) - 4096 and cgm.MAX_NNZ == big - 1
    b = ctypes.c_size_t(0)
    h = ctypes.c_void_p()
    assert L.cogdl_spmm(2, 2, big, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == TOO_LARGE
    assert L.cogdl_spmm_t(2, 2, big, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == TOO_LARGE
    assert L.cogdl_csr_to_csc_workspace(10, 10, big, ctypes.byref(b)) == TOO_LARGE
    assert L.cogdl_csr_to_csc_workspace(10, 10, big - 1, ctypes.byref(b)) == OK
    assert L.cogdl_plan_create(4, big, FAKE, 16, 0, 0, 0, None, ctypes.byref(h)) == TOO_LARGE
    assert L.cogdl_sddmm_dot(2, 2, big, FAKE, FAKE, 2, 4, FAKE, 0, FAKE, 0, FAKE, None, None) == TOO_LARGE
    assert L.cogdl_sddmm_edge_softmax(2, 2, big, FAKE, FAKE, 2, FAKE, FAKE, ctypes.c_float(0.2), FAKE,
                                      None, None) == TOO_LARGE


def test_trace_filter_validation(L):
    # the filter is host state only: no device is touched
    L.cogdl_trace_filter.argtypes = [ctypes.c_char_p]
    assert L.cogdl_trace_filter(b"spmm,gat") == 0
    assert L.cogdl_trace_filter(b"x" * 64) == 1          # a name longer than 63 characters
    assert L.cogdl_trace_filter(b"a," * 600) == 1        # a list longer than 1023 characters
    assert L.cogdl_trace_filter(b",,spmm,") == 0         # empty names are skipped
    assert L.cogdl_trace_filter(None) == 0
    assert L.cogdl_trace_filter(b"") == 0


def _p(v):
    return ctypes.c_void_p(v)


FAKE = _p(0x1000)   # never dereferenced: every call below fails validation first


def test_spmm_validation(L):
    # negative sizes
    assert L.cogdl_spmm(-1, 1, 0, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm(1, 1, -1, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm(1, 1, 0, FAKE, FAKE, None, -4, FAKE, 0, FAKE, 0, None, None) == INVALID
    # dtype codes
    assert L.cogdl_spmm(1, 1, 1, FAKE, FAKE, None, 4, FAKE, 3, FAKE, 0, None, None) == DTYPE
    assert L.cogdl_spmm(1, 1, 1, FAKE, FAKE, None, 4, FAKE, 0, FAKE, -1, None, None) == DTYPE
    # null pointers
    assert L.cogdl_spmm(2, 2, 3, None, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm(2, 2, 3, FAKE, None, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm(2, 2, 3, FAKE, FAKE, None, 4, None, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, None, 0, None, None) == INVALID
    # nnz beyond int32 indices
    assert L.cogdl_spmm(2, 2, 1 << 31, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == TOO_LARGE
    # edges but no columns to gather from
    assert L.cogdl_spmm(2, 0, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    # empty work returns OK without touching the device
    assert L.cogdl_spmm(0, 5, 0, None, None, None, 4, None, 0, None, 0, None, None) == OK
    assert L.cogdl_spmm(3, 5, 7, FAKE, FAKE, None, 0, None, 0, None, 0, None, None) == OK


def test_gspmm_validation(L):
    def G(*a, act=0):
        # (n_rows, n_cols, nnz, rowptr, col, val, F, X, x_dt, Y, y_dt, reduce, compute)
        return L.cogdl_gspmm(*a, None, act, None, None, None)
    # activation codes outside none / relu / elu
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 0, 0, act=3) == INVALID
    # reduce codes outside sum / mean / max, compute codes outside mul / add / sub / copy
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 3, 0) == INVALID
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, -1, 0) == INVALID
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 0, 4) == INVALID
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 2, -1) == INVALID
    # max keeps the input format or widens to fp32: bf16 -> fp16 is refused
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 1, FAKE, 2, 2, 0) == DTYPE
    # fp32 -> bf16 is refused for max, but not for sum / mean (those fail later, on nulls)
    assert G(2, 2, 3, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 1, 2, 1) == DTYPE
    assert G(2, 2, 3, FAKE, None, None, 4, FAKE, 0, FAKE, 1, 1, 2) == INVALID
    # the checks shared with cogdl_spmm
    assert G(-1, 1, 0, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 1, 0) == INVALID
    assert G(2, 2, 1 << 31, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, 2, 3) == TOO_LARGE
    assert G(2, 2, 3, FAKE, FAKE, None, 4, None, 0, FAKE, 0, 2, 0) == INVALID
    assert G(0, 5, 0, None, None, None, 4, None, 0, None, 0, 2, 1) == OK


def test_spmm_t_validation(L):
    assert L.cogdl_spmm_t(3, -2, 0, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID
    assert L.cogdl_spmm_t(3, 2, 5, FAKE, FAKE, None, 4, FAKE, 7, FAKE, 0, None, None) == DTYPE
    assert L.cogdl_spmm_t(0, 2, 5, FAKE, FAKE, None, 4, FAKE, 0, FAKE, 0, None, None) == INVALID


def test_csc_validation(L):
    b = ctypes.c_size_t()
    assert L.cogdl_csr_to_csc_workspace(10, 10, 100, ctypes.byref(b)) == OK
    small = b.value
    assert L.cogdl_csr_to_csc_workspace(10, 10, 100000, ctypes.byref(b)) == OK
    assert b.value > small
    assert L.cogdl_csr_to_csc_workspace(10, 10, -1, ctypes.byref(b)) == INVALID
    assert L.cogdl_csr_to_csc_workspace(10, 10, 1 << 31, ctypes.byref(b)) == TOO_LARGE
    assert L.cogdl_csr_to_csc_workspace(10, 10, 5, None) == INVALID
    ws = _p(0x10000)
    # workspace too small / misaligned / missing
    assert L.cogdl_csr_to_csc(4, 4, 8, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, ws, 16, None) == INVALID
    assert L.cogdl_csr_to_csc(4, 4, 8, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, _p(0x10010),
                              1 << 30, None) == INVALID
    assert L.cogdl_csr_to_csc(4, 4, 8, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, None, 1 << 30,
                              None) == INVALID
    # val and val_t must be given together
    assert L.cogdl_csr_to_csc(4, 4, 8, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws, 1 << 30,
                              None) == INVALID
    assert L.cogdl_csr_to_csc(4, 4, 8, FAKE, FAKE, None, None, FAKE, None, FAKE, ws, 1 << 30,
                              None) == INVALID


def _noalloc_limit():
    m = re.search(r"#define COGDL_NOALLOC_SCRATCH_BYTES \((\d+)ull << (\d+)\)", open(HEADER).read())
    return int(m.group(1)) << int(m.group(2))


def test_csc_noalloc_validation(L):
    """The allocation-free transpose refuses graphs whose workspace exceeds its static scratch,
    and bad arguments, on the host (nothing touches the device)."""
    limit = _noalloc_limit()
    assert limit == 64 << 20
    b = ctypes.c_size_t()
    lo, hi = 1, 1 << 24                      # largest nnz whose workspace fits the scratch
    while lo < hi:
        mid = (lo + hi + 1) // 2
        assert L.cogdl_csr_to_csc_workspace(10, 10, mid, ctypes.byref(b)) == OK
        lo, hi = (mid, hi) if b.value <= limit else (lo, mid - 1)
    assert 1_500_000 < lo < 1_800_000        # "about 1.6M edges", as the header says
    nz = lo + 1
    assert L.cogdl_csr_to_csc_noalloc(10, 10, nz, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, None) == TOO_LARGE
    assert L.cogdl_csr_to_csc_noalloc(10, 10, _max_nnz() + 1, FAKE, FAKE, None, FAKE, FAKE, None, FAKE,
                                      None) == TOO_LARGE
    assert L.cogdl_csr_to_csc_noalloc(-1, 10, 8, FAKE, FAKE, None, FAKE, FAKE, None, FAKE, None) == INVALID
    assert L.cogdl_csr_to_csc_noalloc(4, 4, 8, FAKE, FAKE, None, None, FAKE, None, FAKE, None) == INVALID
    assert L.cogdl_csr_to_csc_noalloc(4, 4, 8, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, None) == INVALID
    assert L.cogdl_csr_to_csc_noalloc(4, 4, 8, FAKE, None, None, FAKE, FAKE, None, FAKE, None) == INVALID


def test_attention_validation(L):
    s = ctypes.c_float(0.2)
    # head count bounds
    assert L.cogdl_sddmm_edge_softmax(4, 4, 8, FAKE, FAKE, 0, FAKE, FAKE, s, FAKE, None, None) == INVALID
    assert L.cogdl_sddmm_edge_softmax(4, 4, 8, FAKE, FAKE, 65, FAKE, FAKE, s, FAKE, None, None) == INVALID
    assert L.cogdl_sddmm_edge_softmax(4, 4, 8, FAKE, FAKE, 2, None, FAKE, s, FAKE, None, None) == INVALID
    assert L.cogdl_sddmm_edge_softmax(4, 4, 8, FAKE, FAKE, 2, FAKE, FAKE, s, None, None, None) == INVALID
    assert L.cogdl_gat_aggregate(4, 4, 8, FAKE, FAKE, 2, 0, FAKE, FAKE, s, None, FAKE, 0, FAKE, 0,
                                 None, None, None) == INVALID
    assert L.cogdl_gat_aggregate(4, 4, 8, FAKE, FAKE, 2, 4, FAKE, FAKE, s, None, FAKE, 5, FAKE, 0,
                                 None, None, None) == DTYPE
    # scores needed unless alpha_in is given
    assert L.cogdl_gat_aggregate(4, 4, 8, FAKE, FAKE, 2, 4, None, FAKE, s, None, FAKE, 0, FAKE, 0,
                                 None, None, None) == INVALID
    assert L.cogdl_gat_aggregate(4, 4, 8, FAKE, FAKE, 2, 4, FAKE, FAKE, s, None, None, 0, FAKE, 0,
                                 None, None, None) == INVALID
    assert L.cogdl_gat_aggregate(0, 4, 0, None, None, 2, 4, None, None, s, None, None, 0, None, 0,
                                 None, None, None) == OK


def test_plan_validation(L):
    h = ctypes.c_void_p()
    assert L.cogdl_plan_create(4, 8, FAKE, 16, 0, 0, 0, None, None) == INVALID
    assert L.cogdl_plan_create(-1, 8, FAKE, 16, 0, 0, 0, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 8, FAKE, 0, 0, 0, 0, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 8, FAKE, 16, 65, 0, 0, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 8, FAKE, 16, 0, 3, 0, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 8, FAKE, 16, 0, 0, -5, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 8, None, 16, 0, 0, 0, None, ctypes.byref(h)) == INVALID
    assert L.cogdl_plan_create(4, 1 << 31, FAKE, 16, 0, 0, 0, None, ctypes.byref(h)) == TOO_LARGE
    assert L.cogdl_plan_destroy(None) == OK
    assert L.cogdl_plan_rebuild(None, FAKE, None) == INVALID
    assert L.cogdl_plan_query(None, None, None) == INVALID
    assert L.cogdl_plan_units(None, FAKE, 4, None) == INVALID


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(3, 4)
    with pytest.raises(cg.CogdlError):
        cg.spmm(torch.zeros(4, dtype=torch.int32), torch.zeros(0, dtype=torch.int32), None, x)


def test_sddmm_dot_validation(L):
    S = L.cogdl_sddmm_dot
    # heads and width
    assert S(2, 2, 3, FAKE, FAKE, 0, 4, FAKE, 0, FAKE, 0, FAKE, None, None) == INVALID
    assert S(2, 2, 3, FAKE, FAKE, 65, 4, FAKE, 0, FAKE, 0, FAKE, None, None) == INVALID
    assert S(2, 2, 3, FAKE, FAKE, 2, 0, FAKE, 0, FAKE, 0, FAKE, None, None) == INVALID
    assert S(2, 2, 3, FAKE, FAKE, 2, 4, FAKE, 5, FAKE, 0, FAKE, None, None) == DTYPE
    assert S(2, 2, 3, FAKE, FAKE, 2, 4, None, 0, FAKE, 0, FAKE, None, None) == INVALID
    assert S(2, 2, 3, FAKE, FAKE, 2, 4, FAKE, 0, FAKE, 0, None, None, None) == INVALID
    assert S(2, 2, 1 << 31, FAKE, FAKE, 2, 4, FAKE, 0, FAKE, 0, FAKE, None, None) == TOO_LARGE
    assert S(0, 3, 0, None, None, 2, 4, None, 0, None, 0, None, None, None) == OK


def test_gat_backward_validation(L):
    def B(n_rows, n_cols, nnz, H=2, D=4, xdt=0, ydt=0, dxdt=0, colptr=FAKE, perm=FAKE, alpha=FAKE,
          dscore=FAKE, ds_src=FAKE, work=FAKE):
        return L.cogdl_gat_backward(n_rows, n_cols, nnz, FAKE, FAKE, colptr, FAKE, perm, H, D, FAKE,
                                    FAKE, ctypes.c_float(0.2), alpha, FAKE, xdt, FAKE, ydt, FAKE, dxdt,
                                    FAKE, dscore, FAKE, ds_src, work, None, None, None)
    assert B(2, 2, 3, H=0) == INVALID
    assert B(2, 2, 3, D=0) == INVALID
    assert B(2, 2, 3, xdt=4) == DTYPE
    assert B(2, 2, 3, dxdt=-1) == DTYPE
    assert B(2, 2, 3, colptr=None) == INVALID
    assert B(2, 2, 3, perm=None) == INVALID
    assert B(2, 2, 3, alpha=None) == INVALID
    # dscore (like dalpha) may be NULL; the missing workspace is what is refused here
    assert B(2, 2, 3, dscore=None, work=None) == INVALID
    assert B(2, 2, 3, ds_src=None) == INVALID
    assert B(2, 2, 3, work=None) == INVALID
    assert B(2, 2, 3, work=_p(0x1004)) == INVALID        # the edge records are 8-byte pairs
    assert B(2, 2, 1 << 31) == TOO_LARGE
    assert B(-1, 2, 0) == INVALID


def test_gat_stats_entry_points_validation(L):
    """The training pair: the forward that writes row softmax states instead of alpha, and the
    backward that rebuilds the weights from them (only failing calls are made)."""
    def F(n_rows=2, n_cols=2, nnz=3, s_src=FAKE, a_src=None, stats=FAKE, act=0):
        return L.cogdl_gat_aggregate_stats(n_rows, n_cols, nnz, FAKE, FAKE, 2, 8, FAKE, s_src, a_src,
                                           ctypes.c_float(0.2), FAKE, 0, FAKE, 0, stats, None, act, None,
                                           None)
    assert F(s_src=None, a_src=None) == INVALID          # exactly one source of scores
    assert F(s_src=FAKE, a_src=FAKE) == INVALID
    assert F(stats=None) == INVALID
    assert F(act=7) == INVALID
    assert F(nnz=1 << 31) == TOO_LARGE

    def B(row_stats=FAKE, work=FAKE, H=2):
        return L.cogdl_gat_backward_stats(2, 2, 3, FAKE, FAKE, FAKE, FAKE, FAKE, H, 4, FAKE, FAKE,
                                          ctypes.c_float(0.2), row_stats, FAKE, 0, FAKE, 0, FAKE, 0,
                                          None, None, FAKE, FAKE, work, None, None, None)
    assert B(row_stats=None) == INVALID
    assert B(work=None) == INVALID
    assert B(H=0) == INVALID


def test_linear_and_head_scores_validation(L):
    lin = L.cogdl_linear
    # n, k, m, X, W, dtype, bias, act, Y, y_dtype, stream
    assert lin(-1, 4, 4, FAKE, FAKE, 1, None, 0, FAKE, 1, None) == INVALID
    assert lin(8, 4, 4, FAKE, FAKE, 0, None, 0, FAKE, 1, None) == DTYPE     # fp32 operands
    assert lin(8, 4, 4, FAKE, FAKE, 1, None, 0, FAKE, 7, None) == DTYPE
    assert lin(8, 4, 4, FAKE, FAKE, 1, None, 5, FAKE, 1, None) == INVALID
    assert lin(8, 4, 4, None, FAKE, 1, None, 0, FAKE, 1, None) == INVALID
    assert lin(8, 4, 4, FAKE, None, 1, None, 0, FAKE, 1, None) == INVALID
    assert lin(8, 4, 4, FAKE, FAKE, 1, None, 0, None, 1, None) == INVALID
    assert lin(0, 4, 4, None, FAKE, 1, None, 0, None, 1, None) == OK
    hs = L.cogdl_head_scores
    # n, H, D, Z, z_dtype, a_src, a_dst, s_src, s_dst, stream
    assert hs(4, 0, 8, FAKE, 1, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    assert hs(4, 2, 0, FAKE, 1, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    assert hs(4, 2, 8, FAKE, 9, FAKE, FAKE, FAKE, FAKE, None) == DTYPE
    assert hs(4, 2, 8, FAKE, 1, None, FAKE, FAKE, FAKE, None) == INVALID
    assert hs(4, 2, 8, None, 1, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    assert hs(4, 2, 8, FAKE, 1, None, None, None, None, None) == OK


def test_codec_validation(L):
    w, s = ctypes.c_int64(), ctypes.c_int64()
    assert L.cogdl_act_codec_size(10, 100, 3, 64, ctypes.byref(w), ctypes.byref(s)) == OK
    assert (w.value, s.value) == (10 * 2 * 1 * 3, 10 * 2 * 2)
    assert L.cogdl_act_codec_size(10, 256, 2, 128, ctypes.byref(w), ctypes.byref(s)) == OK
    assert (w.value, s.value) == (10 * 2 * 2 * 2, 10 * 2 * 2)
    for bits, group in ((0, 64), (9, 64), (2, 32), (2, 96 + 1), (2, 0)):
        assert L.cogdl_act_codec_size(10, 64, bits, group, ctypes.byref(w), ctypes.byref(s)) == INVALID
    C = L.cogdl_act_compress
    assert C(4, 64, FAKE, 5, 2, 64, ctypes.c_uint64(1), FAKE, FAKE, None) == DTYPE
    assert C(4, 0, FAKE, 0, 2, 64, ctypes.c_uint64(1), FAKE, FAKE, None) == INVALID
    assert C(4, 64, None, 0, 2, 64, ctypes.c_uint64(1), FAKE, FAKE, None) == INVALID
    assert C(0, 64, None, 0, 2, 64, ctypes.c_uint64(1), None, None, None) == OK
    D = L.cogdl_act_decompress
    assert D(4, 64, 2, 64, FAKE, FAKE, FAKE, 3, None) == DTYPE
    assert D(4, 64, 2, 64, None, FAKE, FAKE, 0, None) == INVALID


def test_missing_library_fails_loudly(monkeypatch):
    """No CPU fallback: without the HIP library every entry point of the binding raises."""
    import torch
    monkeypatch.setattr(cg, "_lib", None)
    monkeypatch.setattr(cg, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libcogdl_mi355.so"))
    with pytest.raises(cg.CogdlError, match="missing"):
        cg.lib()
    rowptr = torch.zeros(3, dtype=torch.int32)
    col = torch.zeros(0, dtype=torch.int32)
    with pytest.raises(Exception):
        cg.spmm(rowptr, col, None, torch.zeros((2, 4)))


def test_sliced_plan_validation(L):
    """Column-sliced plans: bad arguments are refused before anything is allocated."""
    h = ctypes.c_void_p()
    P = ctypes.c_void_p
    args = dict(n_rows=4, nnz=8, rowptr=FAKE, col=FAKE, n_cols=4, max_feat=8, max_heads=0, mode=0,
                group_size=0, slice_min=0)

    def create(**kw):
        a = dict(args, **kw)
        return L.cogdl_plan_create_sliced(a["n_rows"], a["nnz"], a["rowptr"], a["col"], a["n_cols"],
                                          a["max_feat"], a["max_heads"], a["mode"], a["group_size"],
                                          a["slice_min"], None, ctypes.byref(h))
    assert create(col=None) == INVALID
    assert create(n_cols=0) == INVALID
    assert create(n_cols=-1) == INVALID
    assert create(slice_min=-1) == INVALID
    assert create(group_size=(1 << 24) + 1) == INVALID
    assert create(max_feat=0) == INVALID
    assert create(mode=7) == INVALID
    assert create(nnz=_max_nnz() + 1) == TOO_LARGE
    assert L.cogdl_plan_create_sliced(4, 8, FAKE, FAKE, 4, 8, 0, 0, 0, 0, None, None) == INVALID
    assert L.cogdl_plan_rebuild_sliced(None, FAKE, FAKE, None) == INVALID
    assert L.cogdl_plan_rebuild(None, FAKE, None) == INVALID
    del P
