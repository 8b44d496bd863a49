"""The parity checker itself (tests/compare.py), on hand-made CPU tensors.

Every GPU parity verdict goes through compare(), so it must fail on each
kind of disagreement the tolerance does not cover: an infinity where the
oracle is finite (overflow, a zero divisor), infinities of opposite sign, a
NaN on one side only; and it must accept what the definition leaves equal
(+0 and -0, matching infinities and NaNs, errors at the tolerance)."""
import numpy as np
import pytest
import torch

from compare import compare

INF = float("inf")
NAN = float("nan")


def f32(vals):
    return torch.tensor(vals, dtype=torch.float32)


def test_f32_gpu_inf_where_oracle_finite_fails():
    r = compare(f32([0.25, INF, 0.25]), [0.25, 0.5, 0.25], "f32")
    assert not r["ok"] and r["inf_mismatch"] == 1


def test_f32_gpu_minus_inf_where_oracle_finite_fails():
    assert not compare(f32([-INF, 0.5]), [0.5, 0.5], "f32")["ok"]


def test_f32_gpu_finite_where_oracle_inf_fails():
    assert not compare(f32([1.0, 3.0e38]), [1.0, INF], "f32")["ok"]


def test_f32_opposite_infinities_fail():
    r = compare(f32([1.0, -INF]), [1.0, INF], "f32")
    assert not r["ok"] and r["inf_mismatch"] == 1


def test_f32_matching_infinities_pass():
    r = compare(f32([INF, -INF, 0.5]), [INF, -INF, 0.5], "f32")
    assert r["ok"] and r["max_abs"] == 0.0


@pytest.mark.parametrize("gpu,ref", [([NAN, 1.0], [0.5, 1.0]), ([0.5, 1.0], [NAN, 1.0])])
def test_f32_nan_on_one_side_fails(gpu, ref):
    r = compare(f32(gpu), ref, "f32")
    assert not r["ok"] and r["nan_mismatch"] == 1


def test_f32_nan_against_nan_passes():
    assert compare(f32([NAN, 1.0]), [NAN, 1.0], "f32")["ok"]


def test_f32_signed_zeros_are_equal():
    assert compare(f32([-0.0, 0.0]), [0.0, -0.0], "f32")["ok"]


def test_f32_tolerance_edge():
    # 0.5 + 2^-19 and 0.5 + 2^-20 are exact in fp32; an error of
    # 2^-19 (1.9e-6) fails, 2^-20 (9.5e-7) passes.
    assert not compare(f32([0.5 + 2.0 ** -19]), [0.5], "f32")["ok"]
    r = compare(f32([0.5 + 2.0 ** -20]), [0.5], "f32")
    assert r["ok"] and r["max_abs"] == 2.0 ** -20


def bits16(vals, dtype):
    return torch.tensor(vals, dtype=dtype)


@pytest.mark.parametrize("dtype,fmt,big", [(torch.bfloat16, "bf16", 3.3895e38), (torch.float16, "f16", 65504.0)])
def test_16bit_inf_where_oracle_is_largest_finite_fails(dtype, fmt, big):
    # +inf and the largest finite value are one step apart in the ordered
    # encoding, so only the explicit infinity check catches this.
    r = compare(bits16([1.0, INF], dtype), [1.0, big], fmt)
    assert not r["ok"] and r["inf_mismatch"] == 1


@pytest.mark.parametrize("dtype,fmt", [(torch.bfloat16, "bf16"), (torch.float16, "f16")])
def test_16bit_infinities(dtype, fmt):
    assert compare(bits16([INF, -INF], dtype), [INF, -INF], fmt)["ok"]
    assert not compare(bits16([INF], dtype), [-INF], fmt)["ok"]
    assert not compare(bits16([0.5], dtype), [INF], fmt)["ok"]


@pytest.mark.parametrize("dtype,fmt", [(torch.bfloat16, "bf16"), (torch.float16, "f16")])
def test_16bit_nan_and_zeros(dtype, fmt):
    assert not compare(bits16([NAN], dtype), [0.5], fmt)["ok"]
    assert not compare(bits16([0.5], dtype), [NAN], fmt)["ok"]
    assert compare(bits16([NAN], dtype), [NAN], fmt)["ok"]
    assert compare(bits16([-0.0, 0.0], dtype), [0.0, -0.0], fmt)["ok"]


def test_bf16_ulp_bound():
    one = torch.tensor([1.0], dtype=torch.bfloat16)
    up1 = (one.view(torch.int16) + 1).view(torch.bfloat16)
    up2 = (one.view(torch.int16) + 2).view(torch.bfloat16)
    assert compare(up1, [1.0], "bf16")["ok"]
    r = compare(up2, [1.0], "bf16")
    assert not r["ok"] and r["max_ulp"] == 2 and r["strict_violations"] == 1


def test_floor_rescues_small_values_only():
    # Oracle 1e-7 rounds to a bf16 whose ulp is ~4e-10; the GPU value 2e-7
    # is hundreds of ulps away but within the 2^-22 absolute floor.
    g = torch.tensor([2e-7], dtype=torch.bfloat16)
    assert not compare(g, [1e-7], "bf16")["ok"]
    r = compare(g, [1e-7], "bf16", floor=(2.0 ** -19, 2.0 ** -22))
    assert r["ok"] and r["floor_hits"] == 1 and r["strict_violations"] == 1
    # The floor never rescues an infinity.
    assert not compare(torch.tensor([INF], dtype=torch.bfloat16), [1e-7], "bf16",
                       floor=(2.0 ** -19, 2.0 ** -22))["ok"]


def test_shape_is_flattened_consistently():
    g = f32([[0.0, 1.0], [2.0, 3.0]])
    assert compare(g, np.array([[0.0, 1.0], [2.0, 3.0]]), "f32")["ok"]
    assert not compare(g, np.array([[0.0, 1.0], [3.0, 2.0]]), "f32")["ok"]
