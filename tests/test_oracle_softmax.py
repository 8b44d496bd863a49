"""Pins for the oracle's softmax against facts fixed outside it: closed
forms, invariants, special values, 50-digit brute force and torch's own
float64 CPU softmax (an independent library routine).  The operator is the
PyTorch softmax that the paper validates generated kernels against
(Section III-C)."""
import math
from decimal import Decimal, getcontext

import numpy as np
import pytest
import torch

from oracle import oracle

RNG = np.random.default_rng(1234)


@pytest.mark.parametrize("length", [1, 2, 4, 64, 256, 1024, 4096])
@pytest.mark.parametrize("value", [0.0, -3.5, 1000.0, -1e4])
def test_uniform_row_is_exactly_one_over_length(length, value):
    x = np.full((3, length), value)
    y = oracle.softmax(x)
    assert np.all(y == 1.0 / length)


@pytest.mark.parametrize("offset", [0.0, 1000.0, -1000.0, 88.7])
def test_two_values_ln2_apart_give_thirds(offset):
    # e^0 : e^ln2 = 1 : 2.  The large offsets overflow exp() unless the row
    # maximum is subtracted first.
    x = np.array([offset, offset + math.log(2.0)])
    y = oracle.softmax(x)
    # Storing offset + ln 2 in a double moves it by up to half an ulp of the
    # offset, which shifts the ratio by about that much.
    tol = 1e-15 + 2 * np.spacing(abs(offset))
    assert abs(y[0] - 1.0 / 3.0) < tol
    assert abs(y[1] - 2.0 / 3.0) < tol


def test_length_two_is_the_logistic_function():
    a = RNG.normal(0, 5, 200)
    b = RNG.normal(0, 5, 200)
    y = oracle.softmax(np.stack([a, b], axis=1))
    expect0 = 1.0 / (1.0 + np.exp(b - a))
    np.testing.assert_allclose(y[:, 0], expect0, rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose(y[:, 1], 1.0 - expect0, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("length,pos", [(1, 0), (5, 0), (5, 4), (4096, 0), (4096, 2047)])
def test_single_finite_entry_is_one_hot(length, pos):
    x = np.full(length, -np.inf)
    x[pos] = 0.37
    y = oracle.softmax(x)
    expect = np.zeros(length)
    expect[pos] = 1.0
    assert np.array_equal(y, expect)
    assert not np.any(np.signbit(y))  # masked entries are +0.0


def test_minus_inf_entries_are_exact_zero():
    x = RNG.normal(size=(4, 33))
    x[:, ::3] = -np.inf
    y = oracle.softmax(x)
    assert np.all(y[:, ::3] == 0.0)
    np.testing.assert_allclose(y.sum(axis=1), 1.0, atol=1e-14)


def test_special_rows_follow_ieee_and_pytorch():
    x = np.array([
        [-np.inf, -np.inf, -np.inf],   # fully masked -> NaN (-inf - -inf)
        [0.0, np.nan, 1.0],            # NaN anywhere -> NaN row
        [0.0, np.inf, 1.0],            # +inf -> inf - inf -> NaN row
        [1.0, 2.0, 3.0],               # ordinary row stays finite
    ])
    y = oracle.softmax(x)
    assert np.all(np.isnan(y[:3]))
    assert np.all(np.isfinite(y[3]))
    ref = torch.softmax(torch.from_numpy(x), -1).numpy()
    assert np.array_equal(np.isnan(ref), np.isnan(y))


@pytest.mark.parametrize("shape", [(7, 1), (5, 257), (3, 1024), (2, 3, 65)])
def test_rows_sum_to_one_and_shift_invariance(shape):
    x = RNG.normal(0, 3, shape)
    y = oracle.softmax(x)
    assert np.max(np.abs(y.sum(axis=-1) - 1.0)) < 1e-13
    y2 = oracle.softmax(x + 17.25)
    assert np.max(np.abs(y2 - y)) < 1e-14
    assert np.all(y >= 0)


def _decimal_softmax(row):
    getcontext().prec = 50
    d = [Decimal(float(v)) for v in row]
    m = max(d)
    e = [(v - m).exp() for v in d]
    s = sum(e)
    return [float(v / s) for v in e]


@pytest.mark.parametrize("length", [1, 2, 3, 5, 7])
def test_matches_fifty_digit_brute_force(length):
    x = RNG.normal(0, 4, (6, length))
    y = oracle.softmax(x)
    for r in range(x.shape[0]):
        ref = _decimal_softmax(x[r])
        for j in range(length):
            # exp() and the subtraction each carry about an ulp; allow a few.
            assert abs(y[r, j] - ref[j]) <= 5e-15 * ref[j] + 1e-300


@pytest.mark.parametrize("shape,dim", [((5, 7), -1), ((5, 7), 0), ((2, 3, 4), 1),
                                       ((3, 4, 5, 6), 2), ((1, 8, 16, 16), -1), ((9,), 0)])
def test_matches_torch_float64_softmax(shape, dim):
    # Distinct rows and a non-square shape catch a transposed or wrong axis.
    x = RNG.normal(0, 3, shape)
    y = oracle.softmax(x, dim)
    ref = torch.softmax(torch.from_numpy(x), dim).numpy()
    assert np.max(np.abs(y - ref)) < 1e-15


def test_zero_d_and_empty():
    assert oracle.softmax(np.array(2.5)).item() == 1.0
    assert oracle.softmax(np.zeros((0, 5))).shape == (0, 5)
