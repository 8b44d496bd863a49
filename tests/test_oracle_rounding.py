"""Pins for the oracle's one-step round-to-nearest-even from double into
bfloat16 and binary16: exhaustive round trips, exact rational nearest-value
search, numpy's direct double->half cast (independent library routine),
ties, the double-rounding trap, overflow and gradual underflow."""
import bisect
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle

RNG = np.random.default_rng(5)


def _bf16_values():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    return bits, oracle.bf16_bits_to_f64(bits)


def test_every_bf16_value_round_trips():
    bits, vals = _bf16_values()
    back = oracle.round_bits(vals, "bf16")
    nan = np.isnan(vals)
    assert np.array_equal(back[~nan], bits[~nan])
    assert np.all(np.isnan(oracle.bf16_bits_to_f64(back[nan])))


def test_every_f16_value_round_trips():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float64)
    back = oracle.round_bits(vals, "f16")
    nan = np.isnan(vals)
    assert np.array_equal(back[~nan], bits[~nan])
    assert np.all(np.isnan(back[nan].view(np.float16)))


def test_f16_matches_numpy_direct_cast():
    v = np.concatenate([RNG.normal(0, 1, 20000), RNG.normal(0, 3e4, 5000),
                        RNG.normal(0, 1e-6, 5000), RNG.normal(0, 1e-8, 2000)])
    with np.errstate(over="ignore"):         # overflow to inf is the expected result
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.round_bits(v, "f16"), ref)


def _nearest_bf16_exact(v, table_vals, table_bits):
    """Exact nearest finite positive bf16 by rational distance, ties to even."""
    a = Fraction(abs(v))
    i = bisect.bisect_left(table_vals, a)
    cands = [k for k in (i - 1, i) if 0 <= k < len(table_vals)]
    best = min(cands, key=lambda k: (abs(table_vals[k] - a), table_bits[k] & 1))
    out = table_bits[best]
    return out | (0x8000 if v < 0 else 0)


def test_bf16_matches_exact_rational_nearest():
    bits, vals = _bf16_values()
    pos = (vals >= 0) & np.isfinite(vals) & (bits < 0x8000)
    order = np.argsort(vals[pos], kind="stable")
    tvals = [Fraction(float(v)) for v in vals[pos][order]]
    tbits = [int(b) for b in bits[pos][order]]
    v = np.concatenate([RNG.normal(0, 1, 3000), RNG.normal(0, 1e-39, 500),
                        RNG.normal(0, 1e30, 500), RNG.uniform(-3, 3, 1000)])
    got = oracle.round_bits(v, "bf16")
    for k in range(v.size):
        assert got[k] == _nearest_bf16_exact(float(v[k]), tvals, tbits), v[k]


def test_bf16_ties_go_to_even_and_no_double_rounding():
    # 1 + 2^-8 is the midpoint of 1 and 1 + 2^-7: tie -> even (1.0).
    assert oracle.round_bits(np.array([1.0 + 2.0 ** -8]), "bf16")[0] == 0x3F80
    # 1 + 3*2^-8 is the midpoint of 1+2^-7 (odd) and 1+2^-6 (even): -> up.
    assert oracle.round_bits(np.array([1.0 + 3 * 2.0 ** -8]), "bf16")[0] == 0x3F82
    # Just above the first midpoint by 2^-40: a double->float->bf16 path
    # collapses it onto the midpoint and rounds down; direct RNE rounds up.
    assert oracle.round_bits(np.array([1.0 + 2.0 ** -8 + 2.0 ** -40]), "bf16")[0] == 0x3F81
    assert oracle.round_bits(np.array([-(1.0 + 2.0 ** -8 + 2.0 ** -40)]), "bf16")[0] == 0xBF81


def test_bf16_overflow_and_underflow():
    bf16_max = (2 - 2.0 ** -7) * 2.0 ** 127
    half_ulp = 2.0 ** (127 - 8)
    r = oracle.round_bits(np.array([bf16_max, bf16_max + half_ulp * 0.999,
                                    bf16_max + half_ulp, 1e39, -1e39]), "bf16")
    assert list(r) == [0x7F7F, 0x7F7F, 0x7F80, 0x7F80, 0xFF80]
    tiny = 2.0 ** -133                          # smallest bf16 subnormal
    r = oracle.round_bits(np.array([tiny, tiny / 2, tiny / 2 * 1.0001, tiny * 1.5,
                                    2.0 ** -126, -0.0, 1e-300]), "bf16")
    assert list(r) == [0x0001, 0x0000, 0x0001, 0x0002, 0x0080, 0x8000, 0x0000]


def test_special_values():
    r = oracle.round_bits(np.array([np.inf, -np.inf, np.nan]), "bf16")
    assert r[0] == 0x7F80 and r[1] == 0xFF80
    assert (r[2] & 0x7F80) == 0x7F80 and (r[2] & 0x7F) != 0


def test_f32_rounding_is_numpy_cast():
    v = RNG.normal(size=100)
    assert np.array_equal(oracle.round_to(v, "f32"), v.astype(np.float32))


@pytest.mark.parametrize("fmt", ["bf16", "f16"])
def test_rounding_is_monotone(fmt):
    v = np.sort(RNG.normal(0, 2, 5000))
    r = oracle.round_bits(v, fmt)
    back = oracle.bf16_bits_to_f64(r) if fmt == "bf16" else r.view(np.float16).astype(np.float64)
    assert np.all(np.diff(back) >= 0)
