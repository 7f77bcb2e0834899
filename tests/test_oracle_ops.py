"""Pins for the oracle's arithmetic (CPU only).

Each check ties the oracle to something other than itself:
  * exhaustive agreement, over every pair of codes (specials and non-canonical
    codes included), with the brute-force reference in bruteforce.py, which
    takes values and special-value semantics from IEEE float64 and rounds by
    searching the sorted list of representable values;
  * agreement with IEEE libraries where the formats coincide with IEEE ones on
    normal numbers (paper, Sec. 3.3: the quantized operators behave as IEEE-754
    ones): (5,10) against binary16, (8,7) against bfloat16, (8,23) against
    binary32;
  * algebraic invariants.
"""
import itertools

import numpy as np
import pytest
import torch

import bruteforce as bf
import oracle as orc


def all_codes(wE, wF):
    return np.arange(1 << (3 + wE + wF), dtype=np.uint64)


def pairs(n):
    a = np.repeat(np.arange(n, dtype=np.uint64), n)
    b = np.tile(np.arange(n, dtype=np.uint64), n)
    return a, b


# Formats of at most 9 bits for every multiplier output width the MAC types use
# (Table 3: "single" wF+1, "extended" 2wF+1), plus the same-width product.
SMALL_MUL = [(wE, wF, wFo) for (wE, wF) in [(2, 1), (3, 2), (4, 2), (4, 3), (5, 1), (5, 2), (5, 3)]
             for wFo in sorted({wF, wF + 1, 2 * wF + 1})]


@pytest.mark.parametrize("wE,wF,wFo", SMALL_MUL)
def test_mul_exhaustive_vs_bruteforce(wE, wF, wFo):
    a, b = pairs(1 << (3 + wE + wF))
    got = orc.mul(a, b, wE, wF, wFo)
    ref = bf.mul(a, b, wE, wF, wFo)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} mismatches, first a={a[bad[0]]:#x} b={b[bad[0]]:#x} " \
                          f"got={got[bad[0]]:#x} ref={ref[bad[0]]:#x}"


# Adder formats up to 10 bits wide: these include the accumulators of the
# 8- and 9-bit MAC types, (5,3) and (5,4).
SMALL_ADD = [(2, 1), (3, 2), (4, 2), (4, 3), (4, 4), (5, 2), (5, 3), (5, 4)]


@pytest.mark.parametrize("wE,wF", SMALL_ADD)
def test_add_exhaustive_vs_bruteforce(wE, wF):
    a, b = pairs(1 << (3 + wE + wF))
    got = orc.add(a, b, wE, wF)
    ref = bf.add(a, b, wE, wF)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} mismatches, first a={a[bad[0]]:#x} b={b[bad[0]]:#x} " \
                          f"got={got[bad[0]]:#x} ref={ref[bad[0]]:#x}"


@pytest.mark.parametrize("wE,wFs,wFd", [(5, 3, 4), (5, 4, 3), (5, 6, 3), (5, 4, 5), (5, 11, 4),
                                         (4, 4, 2), (5, 2, 8)])
def test_convert_exhaustive_vs_bruteforce(wE, wFs, wFd):
    c = all_codes(wE, wFs)
    assert np.array_equal(orc.convert(c, wE, wFs, wFd), bf.convert(c, wE, wFs, wFd))


@pytest.mark.parametrize("wE,wF", [(5, 4), (5, 6), (4, 3)])
def test_relu_exhaustive_vs_bruteforce(wE, wF):
    c = all_codes(wE, wF)
    assert np.array_equal(orc.relu(c, wE, wF), bf.relu(c, wE, wF))


def test_muladd_is_add_of_widened_c_and_product():
    g = np.random.default_rng(5)
    wE, wF = 5, 3
    a, b, c = (g.integers(0, 1 << 11, 200000).astype(np.uint64) for _ in range(3))
    p = bf.mul(a, b, wE, wF, wF + 1)
    cw = bf.convert(c, wE, wF, wF + 1)
    ref = bf.add(cw, p, wE, wF + 1)
    assert np.array_equal(orc.muladd(a, b, c, wE, wF, wF + 1), ref)


def test_random_wider_formats_vs_bruteforce():
    """(5,10) inputs with (5,11) products and sums: random codes, all fields random."""
    g = np.random.default_rng(11)
    n = 400000
    a = g.integers(0, 1 << 18, n).astype(np.uint64)
    b = g.integers(0, 1 << 18, n).astype(np.uint64)
    assert np.array_equal(orc.mul(a, b, 5, 10, 11), bf.mul(a, b, 5, 10, 11))
    a = g.integers(0, 1 << 19, n).astype(np.uint64)
    b = g.integers(0, 1 << 19, n).astype(np.uint64)
    assert np.array_equal(orc.add(a, b, 5, 11), bf.add(a, b, 5, 11))


# ---------------------------------------------------------------------------
# IEEE agreement on normal numbers.

def f16_bits_to_code(h):
    """binary16 bit pattern of a normal number -> (5,10) code (same fields, exn=1)."""
    h = np.asarray(h, dtype=np.uint64)
    return (np.uint64(1) << np.uint64(16)) | h


def f16_normal(h_bits):
    e = (np.asarray(h_bits, np.uint32) >> 10) & 0x1F
    return (e >= 1) & (e <= 30)


def test_binary16_mul_agreement():
    """(5,10) x (5,10) -> (5,10) equals binary16 multiplication wherever the
    IEEE operands and result are normal. The float32 product of two binary16
    numbers is exact, so numpy's float16 product is rounded once."""
    g = np.random.default_rng(1)
    n = 1000000
    ha = g.integers(0, 1 << 16, n).astype(np.uint16)
    hb = g.integers(0, 1 << 16, n).astype(np.uint16)
    keep = f16_normal(ha) & f16_normal(hb)
    ha, hb = ha[keep], hb[keep]
    with np.errstate(all="ignore"):
        hr = (ha.view(np.float16) * hb.view(np.float16)).view(np.uint16)
    exact = ha.view(np.float16).astype(np.float64) * hb.view(np.float16).astype(np.float64)
    # IEEE rounds on its subnormal grid below 2^-14, where this format still has
    # a full binade; compare only where the exact result is in IEEE's normal range
    keep = f16_normal(hr) & (np.abs(exact) >= 2.0 ** -14)
    got = orc.mul(f16_bits_to_code(ha[keep]), f16_bits_to_code(hb[keep]), 5, 10, 10)
    assert keep.sum() > 100000
    assert np.array_equal(got, f16_bits_to_code(hr[keep]))


def test_binary16_add_agreement():
    """(5,10) + (5,10) equals binary16 addition on normal numbers: the exact sum
    is formed in float64 and numpy rounds float64 -> float16 once."""
    g = np.random.default_rng(2)
    n = 1000000
    ha = g.integers(0, 1 << 16, n).astype(np.uint16)
    hb = g.integers(0, 1 << 16, n).astype(np.uint16)
    # half of the pairs with nearby exponents, so that cancellation is common
    hb[: n // 2] = (ha[: n // 2] ^ (g.integers(0, 1 << 12, n // 2).astype(np.uint16))) | \
        (g.integers(0, 2, n // 2).astype(np.uint16) << 15)
    keep = f16_normal(ha) & f16_normal(hb)
    ha, hb = ha[keep], hb[keep]
    s = ha.view(np.float16).astype(np.float64) + hb.view(np.float16).astype(np.float64)
    hr = s.astype(np.float16).view(np.uint16)
    keep = f16_normal(hr) & (np.abs(s) >= 2.0 ** -14)
    got = orc.add(f16_bits_to_code(ha[keep]), f16_bits_to_code(hb[keep]), 5, 10)
    assert keep.sum() > 100000
    assert np.array_equal(got, f16_bits_to_code(hr[keep]))


def test_numpy_double_to_half_is_single_rounding():
    # guards the previous test: a double just above a binary16 tie must round up
    # (a detour through float32 would round it to the tie and then to even)
    x = np.float64(1.0 + 2.0 ** -11 + 2.0 ** -40)
    assert float(x.astype(np.float16)) == 1.0 + 2.0 ** -10


def f32_code(bits, extra_exn=True):
    bits = np.asarray(bits, dtype=np.uint64)
    return (np.uint64(1) << np.uint64(32)) | bits


def f32_normal(bits):
    e = (np.asarray(bits, np.uint32) >> 23) & 0xFF
    return (e >= 1) & (e <= 254)


@pytest.mark.parametrize("op", ["mul", "add"])
def test_binary32_agreement(op):
    """(8,23) operations equal the host's IEEE binary32 arithmetic on normal numbers."""
    g = np.random.default_rng(3 if op == "mul" else 4)
    n = 1000000
    a = g.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32)
    if op == "mul":
        b = g.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32)
    else:
        b = a ^ g.integers(0, 1 << 28, n, dtype=np.uint64).astype(np.uint32)
        b ^= (g.integers(0, 2, n).astype(np.uint32) << 31)
    keep = f32_normal(a) & f32_normal(b)
    a, b = a[keep], b[keep]
    fa, fb = a.view(np.float32), b.view(np.float32)
    with np.errstate(all="ignore"):
        r = (fa * fb if op == "mul" else fa + fb).view(np.uint32)
        fa64, fb64 = fa.astype(np.float64), fb.astype(np.float64)
        exact_mag = np.abs(fa64 * fb64 if op == "mul" else fa64 + fb64)  # exact or nearly
    keep = f32_normal(r) & (exact_mag >= 2.0 ** -126)
    assert keep.sum() > 100000
    if op == "mul":
        got = orc.mul(f32_code(a[keep]), f32_code(b[keep]), 8, 23, 23)
    else:
        got = orc.add(f32_code(a[keep]), f32_code(b[keep]), 8, 23)
    assert np.array_equal(got, f32_code(r[keep]))


def bf16_code(bits):
    return (np.uint64(1) << np.uint64(16)) | np.asarray(bits, dtype=np.uint64)


def bf16_normal(bits):
    e = (np.asarray(bits, np.uint32) >> 7) & 0xFF
    return (e >= 1) & (e <= 254)


def test_bfloat16_agreement():
    """(8,7) -> (8,7) equals bfloat16 on normal numbers: products of two bfloat16
    numbers are exact in float32, and so are sums of two whose exponents differ
    by at most 15; torch rounds float32 -> bfloat16 once, to nearest even."""
    g = np.random.default_rng(6)
    n = 1000000
    a = g.integers(0, 1 << 16, n).astype(np.uint16)
    b = g.integers(0, 1 << 16, n).astype(np.uint16)
    b[: n // 2] = (a[: n // 2] & 0x7F80) ^ (g.integers(0, 1 << 11, n // 2).astype(np.uint16)) | \
        (g.integers(0, 2, n // 2).astype(np.uint16) << 15)
    keep = bf16_normal(a) & bf16_normal(b)
    a, b = a[keep], b[keep]
    ta = torch.from_numpy(a.astype(np.int16)).view(torch.bfloat16).float()
    tb = torch.from_numpy(b.astype(np.int16)).view(torch.bfloat16).float()
    for op in ("mul", "add"):
        if op == "mul":
            r32 = ta * tb
            sel = np.ones(len(a), bool)
        else:
            r32 = ta + tb
            ea = (a.astype(np.int32) >> 7) & 0xFF
            eb = (b.astype(np.int32) >> 7) & 0xFF
            sel = np.abs(ea - eb) <= 15
        r = r32.to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
        keep = sel & bf16_normal(r) & np.isfinite(r32.numpy()) & \
            (np.abs(r32.numpy().astype(np.float64)) >= 2.0 ** -126)
        assert keep.sum() > 100000
        if op == "mul":
            got = orc.mul(bf16_code(a[keep]), bf16_code(b[keep]), 8, 7, 7)
        else:
            got = orc.add(bf16_code(a[keep]), bf16_code(b[keep]), 8, 7)
        assert np.array_equal(got, bf16_code(r[keep])), op


# ---------------------------------------------------------------------------
# Special values against IEEE binary32 semantics (library arithmetic).

def test_special_values_follow_ieee_binary32():
    vals = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0, 3.0, -3.0, 0.5],
                    dtype=np.float32)
    a = np.repeat(vals, len(vals))
    b = np.tile(vals, len(vals))
    ca, cb = orc.quantize_f32(a, 8, 23), orc.quantize_f32(b, 8, 23)
    with np.errstate(all="ignore"):
        for op, ref in (("mul", a * b), ("add", a + b)):
            want = orc.quantize_f32(ref, 8, 23)
            got = orc.mul(ca, cb, 8, 23, 23) if op == "mul" else orc.add(ca, cb, 8, 23)
            assert np.array_equal(got, want), op


# ---------------------------------------------------------------------------
# Invariants over random codes of the (5,4) accumulator format.

def test_add_invariants():
    g = np.random.default_rng(7)
    wE, wF = 5, 4
    nb = 3 + wE + wF
    a = g.integers(0, 1 << nb, 300000).astype(np.uint64)
    b = g.integers(0, 1 << nb, 300000).astype(np.uint64)
    sbit = np.uint64(1 << (wE + wF))
    exn = (a >> np.uint64(wE + wF + 1)) & np.uint64(3)
    ab = orc.add(a, b, wE, wF)
    assert np.array_equal(ab, orc.add(b, a, wE, wF))                  # commutative
    canon = orc.add(a, np.uint64(0), wE, wF)                            # a + (+0)
    normal = exn == 1
    assert np.array_equal(canon[normal], a[normal])                     # is a itself
    negsum = orc.add(a ^ sbit, b ^ sbit, wE, wF)                        # (-a) + (-b)
    finite_nonzero = ((ab >> np.uint64(wE + wF + 1)) & np.uint64(3)) == 1
    assert np.array_equal(negsum[finite_nonzero], ab[finite_nonzero] ^ sbit)
    zero_or_nan = orc.add(a, a ^ sbit, wE, wF)                          # a + (-a)
    assert np.all(zero_or_nan[normal] == 0)                             # is +0


def test_rounding_error_at_most_half_ulp():
    g = np.random.default_rng(8)
    wE, wF = 5, 3
    a = (np.uint64(1) << np.uint64(9)) | (g.integers(0, 1 << 9, 200000).astype(np.uint64))
    b = (np.uint64(1) << np.uint64(9)) | (g.integers(0, 1 << 9, 200000).astype(np.uint64))
    p = orc.mul(a, b, wE, wF, wF + 1)
    exact = bf.to_float64(a, wE, wF) * bf.to_float64(b, wE, wF)
    got = bf.to_float64(p, wE, wF + 1)
    ok = np.isfinite(got) & (got != 0)
    ulp = np.ldexp(1.0, (np.floor(np.log2(np.abs(got[ok]))) - (wF + 1)).astype(int))
    assert np.all(np.abs(got[ok] - exact[ok]) <= ulp / 2)
