"""Pins for the oracle's scaled causal softmax (the fused attention-score
softmax: scale, causal mask aligned to the end of the key axis, softmax
over keys): torch's float64 softmax of the explicitly masked scores (an
independent library routine), masked outputs exactly +0, rows summing to 1,
one-hot first rows, a single query row seeing every key, scale folding, and
masked inputs never being read."""
import numpy as np
import pytest
import torch

from oracle import oracle

RNG = np.random.default_rng(77)


def torch_reference(x, scale):
    q, k = x.shape[-2:]
    keep = torch.ones(q, k, dtype=torch.bool).tril(k - q)
    z = torch.from_numpy(x) * scale
    z = z.masked_fill(~keep, float("-inf"))
    return torch.softmax(z, -1).numpy()


@pytest.mark.parametrize("shape", [(4, 4), (2, 3, 16, 16), (1, 5, 7, 12), (3, 1, 9), (2, 6, 6)])
@pytest.mark.parametrize("scale", [1.0, 0.0625, 0.3])
def test_matches_torch_float64_masked_softmax(shape, scale):
    x = RNG.normal(0, 3, shape)
    y = oracle.softmax_causal(x, scale)
    assert np.max(np.abs(y - torch_reference(x, scale))) < 1e-15


def test_masked_entries_are_exact_positive_zero_and_rows_sum_to_one():
    x = RNG.normal(0, 2, (3, 64, 80))
    y = oracle.softmax_causal(x, 0.125)
    q, k = 64, 80
    masked = ~np.tril(np.ones((q, k), dtype=bool), k - q)
    assert np.all(y[:, masked] == 0) and not np.any(np.signbit(y[:, masked]))
    assert np.max(np.abs(y.sum(-1) - 1)) < 1e-13


def test_square_first_row_is_one_hot():
    y = oracle.softmax_causal(RNG.normal(size=(2, 8, 8)), 0.7)
    assert np.all(y[:, 0, 0] == 1.0) and np.all(y[:, 0, 1:] == 0.0)


def test_single_query_row_sees_every_key():
    x = RNG.normal(0, 4, (5, 1, 33))
    assert np.max(np.abs(oracle.softmax_causal(x, 0.25) - oracle.softmax(0.25 * x, -1))) < 1e-16


def test_scale_folds_into_the_input():
    x = RNG.normal(0, 2, (2, 10, 10))
    assert np.array_equal(oracle.softmax_causal(x, 0.5), oracle.softmax_causal(0.5 * x, 1.0))


def test_masked_inputs_are_never_read():
    x = RNG.normal(size=(2, 12, 12))
    poisoned = x.copy()
    poisoned[:, ~np.tril(np.ones((12, 12), dtype=bool))] = np.nan
    assert np.array_equal(oracle.softmax_causal(poisoned, 0.3), oracle.softmax_causal(x, 0.3))


def test_rows_with_no_visible_key_are_nan():
    # More queries than keys: the first q - k rows see nothing (softmax of
    # an all -inf row is NaN, as in PyTorch).
    y = oracle.softmax_causal(RNG.normal(size=(6, 4)), 1.0)
    assert np.all(np.isnan(y[:2])) and np.all(np.isfinite(y[2:]))
