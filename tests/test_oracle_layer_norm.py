"""Pins for the oracle's LayerNorm: torch's float64 CPU layer_norm (an
independent library routine) over several normalised shapes with and
without affine parameters, zero mean and variance v/(v+eps) with identity
affine (biased variance, eps inside the root), constant rows giving the bias
exactly, a two-valued row's closed form, 50-digit brute force, and
agreement with the oracle's GroupNorm at one group (per-channel affine
broadcast over the spatial axes), an independent code path."""
from decimal import Decimal, getcontext

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle

RNG = np.random.default_rng(2024)


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


@pytest.mark.parametrize("shape,nd", [((4, 16), 1), ((2, 3, 1536), 1), ((5, 7), 1), ((2, 4, 6, 8), 2),
                                      ((3, 2, 5, 5), 3), ((1, 1), 1)])
@pytest.mark.parametrize("affine", [True, False])
def test_matches_torch_float64_layer_norm(shape, nd, affine):
    x = RNG.normal(0.3, 1.5, shape)
    ns = shape[len(shape) - nd:]
    w = RNG.normal(1, 0.1, ns) if affine else None
    b = RNG.normal(0, 0.1, ns) if affine else None
    y = oracle.layer_norm(x, nd, w, b, 1e-6)
    ref = F.layer_norm(_t(x), ns, _t(w) if affine else None, _t(b) if affine else None, 1e-6).numpy()
    assert np.max(np.abs(y - ref)) < 1e-13


@pytest.mark.parametrize("eps", [1e-6, 1e-5, 0.25])
def test_identity_affine_moments(eps):
    x = RNG.normal(-2, 3, (6, 257))
    y = oracle.layer_norm(x, 1, None, None, eps)
    v = x.var(axis=-1)
    assert np.max(np.abs(y.mean(axis=-1))) < 1e-14
    np.testing.assert_allclose(y.var(axis=-1), v / (v + eps), rtol=1e-13)


def test_constant_rows_give_bias_exactly():
    x = np.full((3, 10), -1.75)
    b = RNG.normal(size=10)
    assert np.array_equal(oracle.layer_norm(x, 1, RNG.normal(size=10), b, 1e-5), np.broadcast_to(b, x.shape))


def test_two_valued_row_closed_form():
    a, c, eps = 2.0, -1.0, 1e-6
    x = np.array([[a, c, a, c, a, c]])
    half = abs(a - c) / 2
    z = half / np.sqrt(half * half + eps)
    expect = np.where(x == a, z, -z)
    np.testing.assert_allclose(oracle.layer_norm(x, 1, None, None, eps), expect, rtol=1e-15)


def test_matches_fifty_digit_brute_force():
    getcontext().prec = 50
    x = RNG.normal(0.3, 1.5, (3, 7))
    w, b = RNG.normal(1, 0.1, 7), RNG.normal(0, 0.1, 7)
    y = oracle.layer_norm(x, 1, w, b, 1e-6)
    for r in range(3):
        vals = [Decimal(float(v)) for v in x[r]]
        mu = sum(vals) / 7
        var = sum((v - mu) ** 2 for v in vals) / 7
        inv = 1 / (var + Decimal(1e-6)).sqrt()
        for j in range(7):
            ref = float((vals[j] - mu) * inv * Decimal(float(w[j])) + Decimal(float(b[j])))
            assert abs(y[r, j] - ref) < 1e-15


def test_equals_group_norm_with_one_group():
    x = RNG.normal(size=(2, 4, 3, 5))
    w, b = RNG.normal(1, 0.1, 4), RNG.normal(0, 0.1, 4)
    gn = oracle.group_norm(x, 1, w, b, 1e-5)
    ln = oracle.layer_norm(x, 3, np.broadcast_to(w[:, None, None], (4, 3, 5)),
                           np.broadcast_to(b[:, None, None], (4, 3, 5)), 1e-5)
    assert np.max(np.abs(gn - ln)) < 1e-14
