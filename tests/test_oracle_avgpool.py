"""Pins for the oracle's adaptive_avg_pool2d: constant input, identity,
1x1 = plane mean, divisible sizes = fixed-window avg_pool2d, exact rational
brute force, and torch's float64 CPU adaptive_avg_pool2d (independent
library routine).  The operator is PyTorch's adaptive_avg_pool2d, the
reference the paper validates the ResNet-50 pooling kernel against
(Section III-C; Section IV-C, ResNet-50 results)."""
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle

RNG = np.random.default_rng(7)


@pytest.mark.parametrize("hw,out", [((7, 7), (1, 1)), ((13, 17), (5, 7)), ((4, 4), (9, 3))])
@pytest.mark.parametrize("value", [0.375, -1.25, 0.0])
def test_constant_input_gives_constant(hw, out, value):
    # Dyadic constants keep every partial sum exact, so the mean is exact.
    x = np.full((2, 3) + hw, value)
    y = oracle.adaptive_avg_pool2d(x, out)
    assert np.all(y == value)


def test_output_equal_to_input_is_identity():
    x = RNG.normal(size=(2, 3, 6, 5))
    assert np.array_equal(oracle.adaptive_avg_pool2d(x, (6, 5)), x)


@pytest.mark.parametrize("hw", [(1, 1), (7, 7), (8, 8), (14, 14), (3, 11)])
def test_one_by_one_is_plane_mean(hw):
    x = np.maximum(RNG.normal(size=(4, 5) + hw), 0)
    y = oracle.adaptive_avg_pool2d(x, 1)
    np.testing.assert_allclose(y[..., 0, 0], x.mean(axis=(2, 3)), rtol=1e-15, atol=1e-16)


@pytest.mark.parametrize("hw,out", [((8, 8), (2, 2)), ((12, 6), (4, 3)), ((7, 7), (7, 1))])
def test_divisible_sizes_match_fixed_window_pooling(hw, out):
    x = RNG.normal(size=(2, 3) + hw)
    kh, kw = hw[0] // out[0], hw[1] // out[1]
    ref = F.avg_pool2d(torch.from_numpy(x), (kh, kw), (kh, kw)).numpy()
    assert np.max(np.abs(oracle.adaptive_avg_pool2d(x, out) - ref)) < 1e-15


@pytest.mark.parametrize("shape,out", [
    ((2, 3, 7, 7), (1, 1)), ((1, 2, 13, 17), (5, 7)), ((2, 2, 5, 5), (3, 3)),
    ((1, 1, 4, 6), (8, 9)), ((3, 10, 9), (4, 2)), ((1, 3, 1, 1), (2, 3)),
])
def test_matches_torch_float64_adaptive_avg_pool2d(shape, out):
    x = RNG.normal(size=shape)
    ref = F.adaptive_avg_pool2d(torch.from_numpy(x), out).numpy()
    assert np.max(np.abs(oracle.adaptive_avg_pool2d(x, out) - ref)) < 1e-15


def _rational_pool(x, oh, ow):
    h, w = x.shape[-2:]
    planes = x.reshape(-1, h, w)
    out = np.empty((planes.shape[0], oh, ow))
    for p in range(planes.shape[0]):
        for i in range(oh):
            # window rows: every r with floor(i*h/oh) <= r < ceil((i+1)*h/oh)
            rows = [r for r in range(h) if Fraction(i * h, oh) // 1 <= r < -(-Fraction((i + 1) * h, oh) // 1)]
            for j in range(ow):
                cols = [q for q in range(w) if Fraction(j * w, ow) // 1 <= q < -(-Fraction((j + 1) * w, ow) // 1)]
                s = sum(Fraction(float(planes[p, r, q])) for r in rows for q in cols)
                out[p, i, j] = float(s / (len(rows) * len(cols)))
    return out.reshape(x.shape[:-2] + (oh, ow))


@pytest.mark.parametrize("hw,out", [((5, 7), (2, 3)), ((7, 7), (1, 1)), ((3, 4), (5, 6))])
def test_matches_exact_rational_brute_force(hw, out):
    x = RNG.normal(size=(2, 2) + hw)
    y = oracle.adaptive_avg_pool2d(x, out)
    ref = _rational_pool(x, *out)
    # one rounding of the exact mean after a double-precision sum of <= 49 terms
    assert np.max(np.abs(y - ref) / np.maximum(np.abs(ref), 1e-300)) < 1e-14 or \
        np.max(np.abs(y - ref)) < 1e-15
