"""Shared helpers of the GPU parity tests: move seeded inputs to the device,
compare against the oracle with the tolerances of the parity contract."""
from __future__ import annotations

import sys

import numpy as np

from paper_2103_00959_amd import synth

TOL_F32 = 1e-5      # fp32 features: error / Abs (forward-error scale of a sum of products)
TOL_16 = 1e-2       # bf16 / fp16 features or outputs
TOL_ALPHA = 1e-5    # attention weights: plain relative error (alpha > 0)
FLT_MIN = float(np.finfo(np.float32).tiny)

ORACLE_CODE = {"f32": 0, "bf16": 1, "f16": 2}


def say(*a):
    print(*a, flush=True, file=sys.stderr)


def dev(a, dtype=None):
    import torch
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def graph_to_dev(g: synth.Graph):
    return dev(g.rowptr), dev(g.col), dev(g.val)


def features(shape, seed, kind):
    """Host array for the oracle (fp32 values or 16-bit patterns) and the device tensor."""
    import torch
    x = synth.normal_f32(shape, seed)
    if kind == "f32":
        return x, ORACLE_CODE[kind], dev(x)
    if kind == "bf16":
        bits = synth.f32_to_bf16_bits(x)
        return bits, ORACLE_CODE[kind], dev(bits.view(np.int16)).view(torch.bfloat16)
    bits = synth.f32_to_f16_bits(x)
    return bits, ORACLE_CODE[kind], dev(bits.view(np.int16)).view(torch.float16)


def to_f64(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


# significand bits and minimum normal exponent of the output formats
_FORMATS = {"float32": (24, -126), "bfloat16": (8, -126), "float16": (11, -14)}


def half_quantum(y_ref, torch_dtype):
    """Half the spacing of the output format at |y_ref|: the rounding of the
    stored result itself, which dominates near the subnormal range of fp16."""
    p, emin = _FORMATS[str(torch_dtype).replace("torch.", "")]
    e = np.floor(np.log2(np.maximum(np.abs(y_ref), 2.0 ** (emin - p))))
    e = np.maximum(e, emin)
    return 0.5 * np.exp2(e - (p - 1))


def scaled_error(y_gpu, y_ref, abs_ref):
    """max |Y_gpu - Y_ref| / Abs, after allowing the output format's own rounding
    (half a unit in the last place of the stored value)."""
    y = to_f64(y_gpu).reshape(y_ref.shape)
    diff = np.abs(y - y_ref)
    if y_gpu.dtype != __import__("torch").float32:
        diff = np.maximum(diff - half_quantum(y_ref, y_gpu.dtype), 0.0)
    err = diff / np.maximum(abs_ref, 1e-30)
    return float(err.max()) if err.size else 0.0


def tol_for(*kinds):
    return TOL_16 if any(k != "f32" for k in kinds) else TOL_F32


def alpha_close(a_gpu, a_ref, scale=None):
    """Relative error over every weight whose reference is a normal fp32 value, divided by
    `scale` (per weight, default 1): the result must be <= TOL_ALPHA.  Below FLT_MIN (weights
    that underflow in fp32) the absolute error must stay under FLT_MIN."""
    a = to_f64(a_gpu).reshape(a_ref.shape)
    if a_ref.size == 0:
        return 0.0
    normal = a_ref >= FLT_MIN
    assert np.all(np.abs(a[~normal] - a_ref[~normal]) <= FLT_MIN)
    rel = np.abs(a - a_ref) / np.where(normal, a_ref, 1.0)
    if scale is not None:
        rel = rel / scale
    return float(np.max(rel[normal])) if normal.any() else 0.0


def alpha_bound_scale(rowptr, col, sd, ss, slope=0.2, rows=None):
    """The alpha tolerance of the score rounding, as a factor on TOL_ALPHA per weight of the
    edges of `rows` (every row by default), in row order: (1e-5 + 2^-23 max_{k' in row}
    |e_k'|) / 1e-5.  The kernels score an edge in fp32 (e = LeakyReLU(s_dst + s_src) rounded
    once), which moves each weight by at most 2^-24 (|e_k| + max |e_k'|) relative; the
    exponential itself is evaluated to a few units in the last place.  Scores from the fp64
    inputs, per head."""
    rows = np.arange(len(rowptr) - 1) if rows is None else np.asarray(rows)
    deg = (rowptr[rows + 1] - rowptr[rows]).astype(np.int64)
    local = np.repeat(np.arange(rows.size), deg)
    first = np.repeat(np.cumsum(deg) - deg, deg)
    edges = np.repeat(rowptr[rows].astype(np.int64), deg) + (np.arange(int(deg.sum())) - first)
    t = sd[rows[local]].astype(np.float64) + ss[col[edges]].astype(np.float64)
    e = np.where(t > 0, t, slope * t)
    emax = np.zeros((rows.size, sd.shape[1]))
    np.maximum.at(emax, local, np.abs(e))
    return (TOL_ALPHA + 2.0 ** -23 * emax[local]) / TOL_ALPHA
