"""Pins of the oracle's max_pool2d (oracle_max_pool2d in oracle/oracle.c)
against what the definition fixes: torch's float64 CPU max_pool2d (values
and indices) over a sweep of window shapes, strides, paddings, dilations and
ceil mode; an independent brute force in numpy over explicitly enumerated
windows; the output-size formula; closed forms (constant planes, identity
windows, one global window); and the selection rules (first position on a
tie, NaN wins at its last occurrence, all -inf windows)."""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle


def torch_pool(x, k, s, p, d, ceil):
    y, i = F.max_pool2d(torch.from_numpy(x), k, s, p, d, ceil_mode=ceil, return_indices=True)
    return y.numpy(), i.numpy()


CASES = [(k, s, p, d, c) for k in (1, 2, 3, 4) for s in (1, 2, 3) for p in range(k // 2 + 1) for d in (1, 2)
         for c in (False, True)]


@pytest.mark.parametrize("k,s,p,d,ceil", CASES)
def test_matches_torch_float64(k, s, p, d, ceil):
    rng = np.random.default_rng(k * 100 + s * 10 + p + d)
    x = rng.standard_normal((2, 3, 13, 10))
    try:
        ty, ti = torch_pool(x, k, s, p, d, ceil)
    except RuntimeError:
        with pytest.raises(ValueError):
            oracle.max_pool2d(x, k, s, p, d, ceil)
        return
    y, i = oracle.max_pool2d(x, k, s, p, d, ceil)
    assert y.shape == ty.shape
    assert np.array_equal(y, ty) and np.array_equal(i, ti)


def test_rectangular_windows_and_three_d_input():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((5, 17, 12))
    ty, ti = torch_pool(x, (3, 2), (2, 1), (1, 0), (1, 3), True)
    y, i = oracle.max_pool2d(x, (3, 2), (2, 1), (1, 0), (1, 3), True)
    assert np.array_equal(y, ty) and np.array_equal(i, ti)


def brute(x, k, s, p, d, oh, ow):
    """Windows enumerated as explicit coordinate lists; numpy's argmax gives
    the first maximum in row-major window order."""
    planes, h, w = x.shape
    y = np.empty((planes, oh, ow))
    idx = np.empty((planes, oh, ow), dtype=np.int64)
    for pl, i, j in itertools.product(range(planes), range(oh), range(ow)):
        coords = [(i * s - p + a * d, j * s - p + b * d) for a in range(k) for b in range(k)]
        coords = [(r, c) for r, c in coords if 0 <= r < h and 0 <= c < w]
        vals = np.array([x[pl, r, c] for r, c in coords])
        m = int(np.argmax(vals))
        y[pl, i, j] = vals[m]
        idx[pl, i, j] = coords[m][0] * w + coords[m][1]
    return y, idx


@pytest.mark.parametrize("k,s,p,d", [(3, 2, 1, 1), (2, 2, 0, 1), (3, 1, 1, 2), (4, 3, 2, 1)])
def test_brute_force(k, s, p, d):
    rng = np.random.default_rng(11)
    x = rng.standard_normal((3, 11, 9))
    y, i = oracle.max_pool2d(x, k, s, p, d)
    by, bi = brute(x, k, s, p, d, y.shape[1], y.shape[2])
    assert np.array_equal(y, by) and np.array_equal(i, bi)


@pytest.mark.parametrize("n", range(1, 21))
def test_output_size_formula(n):
    for k, s, p, d, c in CASES:
        try:
            t = F.max_pool2d(torch.zeros(1, 1, n, n), k, s, p, d, ceil_mode=c).shape[-1]
        except RuntimeError:
            continue
        assert oracle.pool_out_size(n, k, s, p, d, c) == t, (n, k, s, p, d, c)


def test_resnet_stem_shape():
    x = np.random.default_rng(3).standard_normal((1, 2, 112, 112))
    y, i = oracle.max_pool2d(x, 3, 2, 1)
    ty, ti = torch_pool(x, 3, 2, 1, 1, False)
    assert y.shape == (1, 2, 56, 56) and np.array_equal(y, ty) and np.array_equal(i, ti)


def test_closed_forms():
    c = np.full((2, 7, 6), 0.625)
    y, _ = oracle.max_pool2d(c, 3, 2, 1)
    assert np.all(y == 0.625)
    x = np.random.default_rng(5).standard_normal((2, 7, 6))
    y, i = oracle.max_pool2d(x, 1, 1, 0)                      # identity window
    assert np.array_equal(y, x) and np.array_equal(i[0], np.arange(42).reshape(7, 6))
    y, i = oracle.max_pool2d(x, (7, 6), 1, 0)                 # one global window
    assert y.shape == (2, 1, 1)
    for pl in range(2):
        assert y[pl, 0, 0] == x[pl].max() and i[pl, 0, 0] == int(np.argmax(x[pl]))


def test_selection_rules():
    x = np.zeros((1, 4, 4))
    x[0, 1, 1] = x[0, 1, 2] = 2.0                            # tie: the first position wins
    y, i = oracle.max_pool2d(x, 4, 4, 0)
    assert y[0, 0, 0] == 2.0 and i[0, 0, 0] == 1 * 4 + 1
    x[0, 0, 3] = np.nan
    x[0, 3, 0] = np.nan                                      # NaN wins, at its last occurrence
    y, i = oracle.max_pool2d(x, 4, 4, 0)
    assert np.isnan(y[0, 0, 0]) and i[0, 0, 0] == 3 * 4 + 0
    ninf = np.full((1, 3, 3), -np.inf)                       # all -inf: -inf at the first in-plane position
    y, i = oracle.max_pool2d(ninf, 3, 2, 1)
    assert np.all(y == -np.inf) and i[0, 0, 0] == 0 and i[0, 1, 1] == 1 * 3 + 1
    pos = np.full((1, 3, 3), -1.0)                           # padding is never chosen, even over negatives
    y, i = oracle.max_pool2d(pos, 3, 1, 1)
    assert np.all(y == -1.0) and i[0, 0, 0] == 0


def test_invalid_windows_are_rejected():
    x = np.zeros((1, 5, 5))
    for args in ((3, 1, 2), (0, 1, 0), (2, 0, 0)):
        with pytest.raises(ValueError):
            oracle.max_pool2d(x, *args)
