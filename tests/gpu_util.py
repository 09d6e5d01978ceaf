"""Shared helpers of the GPU parity tests: move seeded inputs to the device,
compare against the oracle with the tolerances of the parity contract."""
from __future__ import annotations

import sys

import numpy as np

from paper_2103_00959_amd import synth

TOL_F32 = 1e-5      # fp32 features: error / Abs (forward-error scale of a sum of products)
TOL_16 = 1e-2       # bf16 / fp16 features or outputs
TOL_ALPHA = 1e-5    # attention weights: plain relative error (alpha > 0)

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
