"""Comparison helpers for parity tests: GPU output vs the float64 oracle.

Both kinds of output: NaN matches only NaN, and an infinity only the same
infinity (an element where exactly one side is infinite, or where the two
infinities differ in sign, fails whatever the tolerance).  fp32 outputs: the
maximum of |gpu - oracle| over the elements finite on both sides.  bf16 /
fp16 outputs: distance in units in the last place between the GPU bits and
the oracle rounded once to the format, counting +0 and -0 as equal.
"""
import sys

import numpy as np
import torch

from oracle import oracle


def note(msg: str):
    """Name the case before a GPU step, flushed, so a crash log shows it."""
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def gpu_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def ordered(bits: np.ndarray) -> np.ndarray:
    """Sign-magnitude 16-bit patterns -> integers whose difference counts
    representable steps (+0 and -0 both map to 0)."""
    mag = (bits & 0x7FFF).astype(np.int64)
    return np.where(bits & 0x8000, -mag, mag)


def _masks(fmt: str) -> tuple:
    return (0x7F80, 0x007F) if fmt == "bf16" else (0x7C00, 0x03FF)


def is_nan_bits(bits: np.ndarray, fmt: str) -> np.ndarray:
    exp_mask, man_mask = _masks(fmt)
    return ((bits & exp_mask) == exp_mask) & ((bits & man_mask) != 0)


def is_inf_bits(bits: np.ndarray, fmt: str) -> np.ndarray:
    exp_mask, man_mask = _masks(fmt)
    return ((bits & exp_mask) == exp_mask) & ((bits & man_mask) == 0)


def compare(gpu: torch.Tensor, ref64: np.ndarray, fmt: str, abs_tol: float = 1e-6, max_ulp: int = 1,
            floor: tuple | None = None) -> dict:
    """Compare a GPU result with the oracle's float64 result.

    fmt "f32": pass if max abs error <= abs_tol.  fmt "bf16"/"f16": pass if
    every element is within max_ulp of the oracle rounded to fmt; with
    floor=(bound, tol), elements whose |oracle| < bound may instead be
    within tol absolutely (reported separately as floor_hits)."""
    ref64 = np.asarray(ref64, dtype=np.float64)
    out = {"fmt": fmt, "n": int(ref64.size)}
    if fmt == "f32":
        g = gpu.detach().float().cpu().numpy().astype(np.float64)
        g, r = g.reshape(-1), ref64.reshape(-1)
        nan_r, nan_g = np.isnan(r), np.isnan(g)
        out["nan_mismatch"] = int(np.count_nonzero(nan_r != nan_g))
        num = ~nan_r & ~nan_g
        inf_any = num & (np.isinf(r) | np.isinf(g))
        out["inf_mismatch"] = int(np.count_nonzero(inf_any & (g != r)))
        both = num & ~inf_any
        err = np.abs(g[both] - r[both])
        out["max_abs"] = float(err.max()) if err.size else 0.0
        out["ok"] = (out["nan_mismatch"] == 0 and out["inf_mismatch"] == 0
                     and out["max_abs"] <= abs_tol)
        return out
    bits = gpu_bits(gpu).reshape(-1)
    ref_bits = oracle.round_bits(ref64, fmt).reshape(-1)
    nan_r, nan_g = is_nan_bits(ref_bits, fmt), is_nan_bits(bits, fmt)
    out["nan_mismatch"] = int(np.count_nonzero(nan_r != nan_g))
    num = ~nan_r & ~nan_g
    inf_any = num & (is_inf_bits(ref_bits, fmt) | is_inf_bits(bits, fmt))
    out["inf_mismatch"] = int(np.count_nonzero(inf_any & (bits != ref_bits)))
    # The largest finite value and infinity are neighbours in the ordered
    # encoding; infinities are settled above, the ulp test covers the rest.
    fin = num & ~inf_any
    dist = np.abs(ordered(bits[fin]) - ordered(ref_bits[fin]))
    bad = dist > max_ulp
    out["max_ulp"] = int(dist.max()) if dist.size else 0
    out["strict_violations"] = int(np.count_nonzero(bad))
    if floor is not None and bad.any():
        bound, tol = floor
        g = (oracle.bf16_bits_to_f64(bits[fin]) if fmt == "bf16"
             else bits[fin].view(np.float16).astype(np.float64))
        r = ref64.reshape(-1)[fin]
        rescued = bad & (np.abs(r) < bound) & (np.abs(g - r) <= tol)
        out["floor_hits"] = int(np.count_nonzero(rescued))
        bad = bad & ~rescued
    out["ok"] = out["nan_mismatch"] == 0 and out["inf_mismatch"] == 0 and not bad.any()
    return out


def assert_close(gpu, ref64, fmt, **kw):
    r = compare(gpu, ref64, fmt, **kw)
    assert r["ok"], r
    return r
