"""Python wrapper around the plain double-precision CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product library
never imports it and it imports nothing from the product package: the two
share no code.

The arithmetic lives in oracle.c; this file only marshals arrays: inputs are
widened exactly to float64 (every bfloat16, binary16 and float32 value is a
double), shapes are flattened to the [rows, len] / [n, c, s] / [planes, h, w]
views the C functions take, and results are rounded once to the output
format.  What each operator computes is PyTorch's definition, which is the
reference the paper validates generated kernels against (Section III-C,
"Kernel Validator").
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# KF_ORACLE_SRC names another copy of oracle.c, built next to it: the pin
# tests use it to check that a mistake planted in the oracle makes them fail.
_SRC = os.environ.get("KF_ORACLE_SRC") or os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(os.path.dirname(os.path.abspath(_SRC)), "liboracle.so")

# Stored significand bits and exponent bits of the narrow output formats.
FORMATS = {"bf16": (7, 8), "f16": (10, 5)}


def compile_oracle(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (no fast-math, no FMA
    contraction, so every operation is one IEEE double rounding)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
            "-fno-fast-math", "-Wall", "-Wextra", "-I", _HERE, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(compile_oracle())
        dp = ctypes.POINTER(ctypes.c_double)
        i64 = ctypes.c_int64
        lib.oracle_softmax_rows.argtypes = [dp, i64, i64, dp]
        lib.oracle_softmax_causal.argtypes = [dp, i64, i64, i64, ctypes.c_double, dp]
        lib.oracle_group_norm.argtypes = [dp, i64, i64, i64, i64, dp, dp, ctypes.c_double, dp]
        lib.oracle_adaptive_avgpool2d.argtypes = [dp, i64, i64, i64, i64, i64, dp]
        lib.oracle_layer_norm.argtypes = [dp, i64, i64, dp, dp, ctypes.c_double, dp]
        lib.oracle_max_pool2d.argtypes = [dp] + [i64] * 13 + [dp, ctypes.POINTER(ctypes.c_int64)]
        lib.oracle_round_to_format.argtypes = [dp, i64, ctypes.c_int, ctypes.c_int,
                                               ctypes.POINTER(ctypes.c_uint32)]
        for f in (lib.oracle_softmax_rows, lib.oracle_softmax_causal, lib.oracle_group_norm,
                  lib.oracle_adaptive_avgpool2d, lib.oracle_layer_norm, lib.oracle_max_pool2d,
                  lib.oracle_round_to_format):
            f.restype = None
        _lib = lib
    return _lib


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a) -> np.ndarray:
    """Exact widening to a C-contiguous float64 array.  Accepts numpy arrays
    or torch CPU tensors (bfloat16 is widened through its bit pattern)."""
    if hasattr(a, "detach"):  # torch tensor
        import torch
        t = a.detach().cpu()
        if t.dtype == torch.bfloat16:
            bits = t.contiguous().view(torch.int16).numpy().astype(np.uint16)
            return bf16_bits_to_f64(bits)
        a = t.numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact: bf16 is the top half of an
    IEEE single)."""
    u32 = bits.astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):     # NaN payloads widen to NaN
        return u32.view(np.float32).astype(np.float64)


def softmax(x, dim: int = -1) -> np.ndarray:
    """PyTorch softmax(x, dim) in float64."""
    x = _f64(x)
    if x.ndim == 0:
        x = x.reshape(1)
        squeeze = True
    else:
        squeeze = False
    dim = dim % x.ndim
    xm = np.ascontiguousarray(np.moveaxis(x, dim, -1))
    length = xm.shape[-1]
    rows = xm.size // length if length else 0
    ym = np.empty_like(xm)
    if xm.size:
        _load().oracle_softmax_rows(_dptr(xm), rows, length, _dptr(ym))
    y = np.moveaxis(ym, -1, dim)
    return np.ascontiguousarray(y.reshape(()) if squeeze else y)


def softmax_causal(x, scale: float = 1.0) -> np.ndarray:
    """Scaled causal softmax over the last axis of x [..., q, k] in float64:
    query i sees keys j <= i + (k - q); masked outputs are +0."""
    x = _f64(x)
    if x.ndim < 2:
        raise ValueError("softmax_causal expects [..., q, k]")
    q, k = x.shape[-2], x.shape[-1]
    batch = x.size // (q * k) if q * k else 0
    y = np.empty_like(x)
    if x.size:
        _load().oracle_softmax_causal(_dptr(x), batch, q, k, float(scale), _dptr(y))
    return y


def group_norm(x, num_groups: int, weight=None, bias=None, eps: float = 1e-5) -> np.ndarray:
    """PyTorch group_norm(x, num_groups, weight, bias, eps) in float64;
    x is [N, C, *]."""
    x = _f64(x)
    if x.ndim < 2:
        raise ValueError("group_norm expects [N, C, *]")
    n, c = x.shape[0], x.shape[1]
    if c % num_groups:
        raise ValueError("C must be divisible by num_groups")
    s = int(np.prod(x.shape[2:], dtype=np.int64)) if x.ndim > 2 else 1
    w = _f64(weight) if weight is not None else None
    b = _f64(bias) if bias is not None else None
    for v in (w, b):
        if v is not None and v.shape != (c,):
            raise ValueError("affine parameters must have shape [C]")
    y = np.empty_like(x)
    if x.size:
        lib = _load()
        null = ctypes.POINTER(ctypes.c_double)()
        lib.oracle_group_norm(_dptr(x), n, c, s, num_groups,
                              _dptr(w) if w is not None else null,
                              _dptr(b) if b is not None else null,
                              float(eps), _dptr(y))
    return y


def layer_norm(x, normalized_ndim: int = 1, weight=None, bias=None, eps: float = 1e-5) -> np.ndarray:
    """PyTorch layer_norm(x, x.shape[-normalized_ndim:], weight, bias, eps)
    in float64; weight / bias have the normalised shape (or are None)."""
    x = _f64(x)
    if not 1 <= normalized_ndim <= x.ndim:
        raise ValueError("normalized_ndim must be in [1, x.ndim]")
    d = int(np.prod(x.shape[x.ndim - normalized_ndim:], dtype=np.int64))
    rows = x.size // d if d else 0
    w = _f64(weight).reshape(-1) if weight is not None else None
    b = _f64(bias).reshape(-1) if bias is not None else None
    for v in (w, b):
        if v is not None and v.size != d:
            raise ValueError("affine parameters must have the normalised shape")
    y = np.empty_like(x)
    if x.size:
        null = ctypes.POINTER(ctypes.c_double)()
        _load().oracle_layer_norm(_dptr(x), rows, d, _dptr(w) if w is not None else null,
                                  _dptr(b) if b is not None else null, float(eps), _dptr(y))
    return y


def adaptive_avg_pool2d(x, output_size) -> np.ndarray:
    """PyTorch adaptive_avg_pool2d(x, output_size) in float64; x is
    [N, C, H, W] or [C, H, W]."""
    x = _f64(x)
    if x.ndim not in (3, 4):
        raise ValueError("adaptive_avg_pool2d expects [N, C, H, W] or [C, H, W]")
    if isinstance(output_size, int):
        oh = ow = output_size
    else:
        oh, ow = output_size
    h, w = x.shape[-2], x.shape[-1]
    planes = int(np.prod(x.shape[:-2], dtype=np.int64))
    y = np.empty(x.shape[:-2] + (oh, ow), dtype=np.float64)
    if y.size:
        _load().oracle_adaptive_avgpool2d(_dptr(x), planes, h, w, oh, ow, _dptr(y))
    return y


def _pair(v):
    return (v, v) if isinstance(v, int) else tuple(v)


def pool_out_size(n: int, k: int, s: int, p: int, d: int, ceil_mode: bool) -> int:
    """Output length of a pooling window sweep (PyTorch's formula): the
    number of window starts i*s - p whose effective extent d*(k-1)+1 fits in
    the padded length, rounded up in ceil mode, where a last window that
    would start inside the right padding is dropped."""
    span = n + 2 * p - d * (k - 1) - 1
    out = (-(-span // s) if ceil_mode else span // s) + 1
    if ceil_mode and (out - 1) * s >= n + p:
        out -= 1
    return out


def max_pool2d(x, kernel_size, stride=None, padding=0, dilation=1, ceil_mode=False):
    """PyTorch max_pool2d(x, ...) with return_indices: (y float64, idx int64)
    for x [N, C, H, W] or [C, H, W] (any memory layout; the logical tensor is
    what is pooled)."""
    x = _f64(x)
    if x.ndim not in (3, 4):
        raise ValueError("max_pool2d expects [N, C, H, W] or [C, H, W]")
    kh, kw = _pair(kernel_size)
    sh, sw = _pair(stride if stride is not None else kernel_size)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    if min(kh, kw, sh, sw, dh, dw) < 1 or min(ph, pw) < 0 or ph > kh // 2 or pw > kw // 2:
        raise ValueError("bad max_pool2d window")
    h, w = x.shape[-2], x.shape[-1]
    oh = pool_out_size(h, kh, sh, ph, dh, ceil_mode)
    ow = pool_out_size(w, kw, sw, pw, dw, ceil_mode)
    if oh < 1 or ow < 1:
        raise ValueError("max_pool2d output would be empty")
    planes = int(np.prod(x.shape[:-2], dtype=np.int64))
    y = np.empty(x.shape[:-2] + (oh, ow), dtype=np.float64)
    idx = np.empty(y.shape, dtype=np.int64)
    if y.size:
        _load().oracle_max_pool2d(_dptr(x), planes, h, w, kh, kw, sh, sw, ph, pw, dh, dw, oh, ow, _dptr(y),
                                  idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    return y, idx


def round_bits(y: np.ndarray, fmt: str) -> np.ndarray:
    """Round float64 values once, to nearest-even, into `fmt` ("bf16" or
    "f16"); returns the uint16 bit patterns."""
    mant, expo = FORMATS[fmt]
    y = np.ascontiguousarray(np.asarray(y, dtype=np.float64))
    out = np.empty(y.shape, dtype=np.uint32)
    if y.size:
        _load().oracle_round_to_format(
            _dptr(y), y.size, mant, expo, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)))
    return out.astype(np.uint16)


def round_to(y: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 results to the output dtype: "f32" gives float32
    (numpy's correctly rounded cast), "bf16"/"f16" give uint16 bits."""
    if dtype == "f32":
        return np.asarray(y, dtype=np.float64).astype(np.float32)
    return round_bits(y, dtype)
