"""Pins for the oracle's global average pooling and its scale factor.

The pooling layer is the one the paper proposes for the interface between
the last convolution and the fully connected layer of MobileNets (Sec. 4):
a sum over the H x W positions in the accumulator format, rounded after every
add, then one multiply by the nearest code of 1/(H W). The pins below do not
use the oracle's own rounding: they use exact rationals, numpy's mean and
the float64 search of tests/bruteforce.py.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from bruteforce import nearest, to_float64

RNE, RTZ = oracle.RNE, oracle.RTZ


def code_value(code, wE, wF):
    """Exact value of a normal code, as a Fraction."""
    code = int(code)
    F = code & ((1 << wF) - 1)
    E = (code >> wF) & ((1 << wE) - 1)
    s = (code >> (wF + wE)) & 1
    assert (code >> (wF + wE + 1)) & 3 == 1, "normal codes only"
    bias = (1 << (wE - 1)) - 1
    v = Fraction((1 << wF) + F) * Fraction(2) ** (E - bias - wF)
    return -v if s else v


def nearest_rational(v, wE, wF):
    """Code of the positive rational v rounded to nearest, ties to the even
    fraction: the two neighbours on the grid of v's binade are compared
    exactly (no exponent range check; the values here are in range)."""
    assert v > 0
    u = 0
    while Fraction(2) ** u > v:
        u -= 1
    while Fraction(2) ** (u + 1) <= v:
        u += 1
    ulp = Fraction(2) ** (u - wF)
    k = v / ulp                      # in [2^wF, 2^(wF+1))
    lo = k.numerator // k.denominator
    rem = k - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    if lo == 1 << (wF + 1):
        lo >>= 1
        u += 1
    bias = (1 << (wE - 1)) - 1
    if u + bias < 0:
        return None                  # below the smallest normal
    return (1 << (wF + wE + 1)) | ((u + bias) << wF) | (lo - (1 << wF))


@pytest.mark.parametrize("wE,wF", [(5, 3), (5, 4), (5, 10), (4, 4), (8, 7)])
def test_recip_is_nearest_code(wE, wF):
    for n in list(range(1, 70)) + [100, 196, 1000, 3136, 12544]:
        want = nearest_rational(Fraction(1, n), wE, wF)
        want = 0 if want is None else want    # flushed to +0 below the range
        assert int(oracle.recip(n, wE, wF)) == want, n


def test_recip_powers_of_two_exact():
    for k in range(0, 14):
        c = oracle.recip(1 << k, 5, 4)
        assert code_value(c, 5, 4) == Fraction(1, 1 << k)


def test_recip_flushes_below_range():
    # (4, 3): bias 7, so the smallest normal is 2^-7; 1/256 flushes to +0
    assert int(oracle.recip(256, 4, 3)) == 0
    assert code_value(oracle.recip(128, 4, 3), 4, 3) == Fraction(1, 128)


def test_single_position_is_a_multiply_by_one():
    g = np.random.default_rng(1)
    x = oracle.quantize_f32(g.normal(size=(3, 1, 1, 40)).astype(np.float32), 5, 4)
    out = oracle.avgpool(x, 5, 4, 4, 4)
    assert np.array_equal(out, x.reshape(3, 40))
    # narrower output: x * 1 rounded once, i.e. converted
    out3 = oracle.avgpool(x, 5, 4, 4, 3)
    assert np.array_equal(out3, nearest(to_float64(x.reshape(3, 40), 5, 4), 5, 3))


@pytest.mark.parametrize("H,W", [(2, 2), (4, 4), (2, 8), (1, 16)])
def test_exact_sums_give_numpy_mean(H, W):
    """Small integers whose partial sums are exact in (6, 12): with H W a power
    of two the scale is exact, so the result is the exact mean."""
    g = np.random.default_rng([2, H, W])
    ints = g.integers(-60, 61, size=(2, H, W, 33)).astype(np.float32)
    x = oracle.quantize_f32(ints, 6, 12)
    out = oracle.avgpool(x, 6, 12, 12, 12)
    want = np.mean(ints.astype(np.float64), axis=(1, 2))
    got = to_float64(out, 6, 12)
    assert np.array_equal(got, want)


def test_exact_sum_then_one_rounding():
    """H W = 49 (the MobileNets 7 x 7 map): with exact partial sums the result
    is the nearest code to (sum) x (nearest code of 1/49), computed here with
    rationals."""
    g = np.random.default_rng(3)
    ints = g.integers(1, 40, size=(1, 7, 7, 8)).astype(np.float32)
    x = oracle.quantize_f32(ints, 6, 12)
    out = oracle.avgpool(x, 6, 12, 12, 5)
    s = code_value(oracle.recip(49, 6, 12), 6, 12)
    for c in range(8):
        total = Fraction(int(ints[0, :, :, c].sum()))
        assert int(out[0, c]) == nearest_rational(total * s, 6, 5), c


def test_order_is_rows_then_columns():
    """(5,3) keeps 4 significant bits, so on 64..127 the grid step is 8 and a
    1 added to 64 is lost. Ones added before a 64 count; ones after it do not.
    A 4 x 4 map of ones with one 64:
      64 last (3,3):  15 ones = 15, + 64 = 79 -> 80; mean 80/16 = 5
      64 first (0,0): 64, then every 1 is lost;     mean 64/16 = 4
      64 at (0,3): rows first, 3 + 64 = 67 -> 64, then lost: mean 4
                   (columns first would be 12 + 64 = 76, a tie -> 80: mean 5)"""
    wE, wF = 5, 3
    for pos, want in [((3, 3), 5.0), ((0, 0), 4.0), ((0, 3), 4.0)]:
        vals = np.ones((1, 4, 4, 1), np.float32)
        vals[0, pos[0], pos[1], 0] = 64.0
        out = oracle.avgpool(oracle.quantize_f32(vals, wE, wF), wE, wF, wF, wF)
        assert to_float64(out, wE, wF)[0, 0] == want, pos


def test_specials():
    wE, wF = 5, 4
    nan, inf = np.nan, np.inf
    rows = np.array([
        [1.0, 2.0, nan, 3.0],     # NaN propagates
        [inf, 1.0, -inf, 2.0],    # +inf + -inf -> NaN
        [inf, 1.0, 2.0, 3.0],     # +inf stays
        [-0.0, -0.0, -0.0, -0.0],  # the sum starts at +0: +0 + -0 = +0
        [1.0, -1.0, 2.0, -2.0],   # exact cancellation -> +0
    ], np.float32).reshape(5, 2, 2, 1)
    out = oracle.avgpool(oracle.quantize_f32(rows, wE, wF), wE, wF, wF, wF)
    v = to_float64(out.reshape(-1), wE, wF)
    assert np.isnan(v[0]) and np.isnan(v[1])
    assert v[2] == inf
    assert v[3] == 0 and not np.signbit(v[3])
    assert v[4] == 0 and not np.signbit(v[4])


def test_rtz_below_the_exact_mean():
    """Positive inputs: every truncated partial sum is at most the exact one,
    so the result is at most (exact sum) x s, s the scale code's value."""
    g = np.random.default_rng(4)
    vals = np.abs(g.normal(size=(2, 7, 7, 16))).astype(np.float32) + 0.01
    x = oracle.quantize_f32(vals, 5, 4)
    out = oracle.avgpool(x, 5, 4, 5, 4, rnd=RTZ)
    s = code_value(oracle.recip(49, 5, 5), 5, 5)
    xv = to_float64(x, 5, 4)
    for n in range(2):
        for c in range(16):
            exact = sum(Fraction(float(v)) for v in xv[n, :, :, c].reshape(-1))
            assert code_value(out[n, c], 5, 4) <= exact * s
    assert not np.array_equal(out, oracle.avgpool(x, 5, 4, 5, 4, rnd=RNE))


def test_rejects_bad_arguments():
    x = np.zeros((1, 2, 2, 3), np.uint64)
    with pytest.raises(ValueError):
        oracle.avgpool(x, 5, 5, 4, 4)     # wF_in > wF_acc
    with pytest.raises(ValueError):
        oracle.recip(0, 5, 4)
