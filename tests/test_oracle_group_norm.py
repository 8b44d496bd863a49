"""Pins for the oracle's GroupNorm: invariants, reductions to instance norm
and layer norm, closed forms for constant and two-valued groups, 50-digit
brute force, and torch's float64 CPU group_norm (independent library
routine).  The operator is PyTorch's group_norm, the reference the paper
validates the SD3.5 group_norm kernel against (Section III-C; Section IV-C,
SD3.5 results)."""
from decimal import Decimal, getcontext

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle

RNG = np.random.default_rng(99)


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


@pytest.mark.parametrize("eps", [1e-6, 1e-5, 0.5])
def test_identity_affine_gives_zero_mean_and_shrunk_variance(eps):
    n, c, h, w, g = 2, 12, 5, 3, 4
    x = RNG.normal(0.3, 1.5, (n, c, h, w))
    y = oracle.group_norm(x, g, None, None, eps)
    xg = x.reshape(n, g, -1)
    yg = y.reshape(n, g, -1)
    v = xg.var(axis=-1)                       # biased variance (numpy, ddof=0)
    assert np.max(np.abs(yg.mean(axis=-1))) < 1e-14
    # Var(y) = v / (v + eps): biased variance, eps inside the square root.
    np.testing.assert_allclose(yg.var(axis=-1), v / (v + eps), rtol=1e-13)


def test_groups_equal_channels_is_instance_norm():
    x = RNG.normal(-1, 2, (3, 6, 4, 5))
    y = oracle.group_norm(x, 6, None, None, 1e-5)
    ref = F.instance_norm(_t(x), eps=1e-5).numpy()
    assert np.max(np.abs(y - ref)) < 1e-13


def test_single_group_is_layer_norm_over_chw():
    x = RNG.normal(0.5, 1, (2, 4, 3, 3))
    w = RNG.normal(1, 0.2, 4)
    b = RNG.normal(0, 0.2, 4)
    y = oracle.group_norm(x, 1, w, b, 1e-6)
    wf = np.broadcast_to(w[:, None, None], (4, 3, 3))
    bf = np.broadcast_to(b[:, None, None], (4, 3, 3))
    ref = F.layer_norm(_t(x), (4, 3, 3), _t(wf.copy()), _t(bf.copy()), 1e-6).numpy()
    assert np.max(np.abs(y - ref)) < 1e-13


def test_constant_group_gives_bias_exactly():
    x = np.full((1, 8, 3, 3), 2.75)
    x[:, 4:] = -0.5                           # second group is another constant
    w = RNG.normal(1, 0.1, 8)
    b = RNG.normal(0, 0.1, 8)
    y = oracle.group_norm(x, 2, w, b, 1e-6)
    assert np.array_equal(y, np.broadcast_to(b[None, :, None, None], y.shape))


@pytest.mark.parametrize("a,bv,eps", [(1.0, 3.0, 1e-6), (-2.5, 0.25, 1e-5), (0.0, 1e-3, 1e-6)])
def test_two_valued_group_closed_form(a, bv, eps):
    # Half the group at a, half at bv: mean (a+bv)/2, variance (a-bv)^2/4.
    x = np.empty((1, 2, 4, 4))
    x[0].reshape(-1)[:16] = a
    x[0].reshape(-1)[16:] = bv
    w = np.array([1.5, -0.75])
    b = np.array([0.25, 0.125])
    y = oracle.group_norm(x, 1, w, b, eps)
    half = abs(a - bv) / 2.0
    z = half / np.sqrt(half * half + eps)
    za = z if a > bv else -z
    expect = np.empty_like(x)
    for ch in range(2):
        flat = expect[0, ch].reshape(-1)
        vals = x[0, ch].reshape(-1)
        flat[:] = np.where(vals == a, za, -za) * w[ch] + b[ch]
    np.testing.assert_allclose(y, expect, rtol=1e-14, atol=1e-15)


def _decimal_group_norm(x, g, w, b, eps):
    getcontext().prec = 50
    n, c = x.shape[:2]
    out = np.empty_like(x)
    cg = c // g
    for i in range(n):
        for k in range(g):
            vals = [Decimal(float(v)) for v in x[i, k * cg:(k + 1) * cg].reshape(-1)]
            cnt = Decimal(len(vals))
            mu = sum(vals) / cnt
            var = sum((v - mu) ** 2 for v in vals) / cnt
            r = 1 / (var + Decimal(eps)).sqrt()
            for ch in range(k * cg, (k + 1) * cg):
                src = x[i, ch].reshape(-1)
                dst = out[i, ch].reshape(-1)
                for j in range(src.size):
                    dst[j] = float((Decimal(float(src[j])) - mu) * r * Decimal(float(w[ch]))
                                   + Decimal(float(b[ch])))
    return out


def test_matches_fifty_digit_brute_force():
    x = RNG.normal(0.3, 1.5, (2, 6, 2, 3))
    w = RNG.normal(1, 0.1, 6)
    b = RNG.normal(0, 0.1, 6)
    y = oracle.group_norm(x, 3, w, b, 1e-6)
    ref = _decimal_group_norm(x, 3, w, b, 1e-6)
    assert np.max(np.abs(y - ref)) < 1e-14


@pytest.mark.parametrize("shape,g,affine", [
    ((2, 8), 4, True),                  # [N, C]: one element per channel
    ((3, 6, 10), 3, False),             # [N, C, L]
    ((2, 16, 4, 4), 4, True),
    ((1, 32, 7, 7), 8, True),
    ((2, 4, 2, 3, 2), 2, True),         # 3-D spatial
    ((1, 512, 4, 4), 32, True),
])
def test_matches_torch_float64_group_norm(shape, g, affine):
    x = RNG.normal(0.3, 1.5, shape)
    c = shape[1]
    w = RNG.normal(1, 0.1, c) if affine else None
    b = RNG.normal(0, 0.1, c) if affine else None
    y = oracle.group_norm(x, g, w, b, 1e-6)
    ref = F.group_norm(_t(x), g, _t(w) if affine else None, _t(b) if affine else None, 1e-6).numpy()
    assert np.max(np.abs(y - ref)) < 1e-13


def test_weight_only_and_bias_only():
    x = RNG.normal(size=(2, 4, 3))
    w = RNG.normal(1, 0.1, 4)
    b = RNG.normal(0, 0.1, 4)
    y_w = oracle.group_norm(x, 2, w, None, 1e-5)
    y_b = oracle.group_norm(x, 2, None, b, 1e-5)
    ref_w = F.group_norm(_t(x), 2, _t(w), None, 1e-5).numpy()
    ref_b = F.group_norm(_t(x), 2, None, _t(b), 1e-5).numpy()
    assert np.max(np.abs(y_w - ref_w)) < 1e-13
    assert np.max(np.abs(y_b - ref_b)) < 1e-13


def test_rejects_indivisible_channels():
    with pytest.raises(ValueError):
        oracle.group_norm(np.zeros((1, 6, 2)), 4)
