"""Pins for the oracle's round-toward-zero mode (CPU only).

The paper's second rounding mode (Sec. 4: round-toward-zero versions of the
MACs). Each check ties the oracle to something other than itself:
  * exhaustive agreement over every pair of small-format codes with the
    brute-force reference (bruteforce.py), which picks the representable value
    of largest magnitude not above the exact value's;
  * agreement with IEEE binary16 on normal results: numpy rounds to nearest,
    and the toward-zero result is that one, or its neighbour toward zero when
    the nearest one lies beyond the exact value;
  * invariants: never larger in magnitude than the exact value nor than the
    nearest-rounded result, equal to it whenever that one is exact, and within
    one unit in the last place.
"""
import numpy as np
import pytest

import bruteforce as bf
import oracle as orc

RTZ = orc.RTZ


def pairs(n):
    return np.repeat(np.arange(n, dtype=np.uint64), n), np.tile(np.arange(n, dtype=np.uint64), n)


@pytest.mark.parametrize("wE,wF,wFo", [(2, 1, 1), (3, 2, 3), (4, 2, 3), (4, 3, 4), (4, 3, 7),
                                        (5, 2, 3), (5, 2, 5), (5, 3, 4)])
def test_mul_rtz_exhaustive_vs_bruteforce(wE, wF, wFo):
    a, b = pairs(1 << (3 + wE + wF))
    got = orc.mul(a, b, wE, wF, wFo, rnd=RTZ)
    ref = bf.mul(a, b, wE, wF, wFo, mode="rtz")
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} mismatches, first a={a[bad[0]]:#x} b={b[bad[0]]:#x}"


@pytest.mark.parametrize("wE,wF", [(2, 1), (3, 2), (4, 3), (5, 2), (5, 3), (5, 4)])
def test_add_rtz_exhaustive_vs_bruteforce(wE, wF):
    a, b = pairs(1 << (3 + wE + wF))
    got = orc.add(a, b, wE, wF, rnd=RTZ)
    ref = bf.add(a, b, wE, wF, mode="rtz")
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} mismatches, first a={a[bad[0]]:#x} b={b[bad[0]]:#x}"


@pytest.mark.parametrize("wE,wFs,wFd", [(5, 4, 3), (5, 6, 3), (5, 11, 4), (5, 3, 4), (4, 7, 3)])
def test_convert_rtz_exhaustive_vs_bruteforce(wE, wFs, wFd):
    c = np.arange(1 << (3 + wE + wFs), dtype=np.uint64)
    assert np.array_equal(orc.convert(c, wE, wFs, wFd, rnd=RTZ),
                          bf.convert(c, wE, wFs, wFd, mode="rtz"))


def test_muladd_rtz_composition():
    g = np.random.default_rng(15)
    wE, wF = 5, 3
    a, b, c = (g.integers(0, 1 << 11, 200000).astype(np.uint64) for _ in range(3))
    ref = bf.add(bf.convert(c, wE, wF, wF + 1, "rtz"), bf.mul(a, b, wE, wF, wF + 1, "rtz"),
                 wE, wF + 1, "rtz")
    assert np.array_equal(orc.muladd(a, b, c, wE, wF, wF + 1, rnd=RTZ), ref)


def f16_code(h):
    return (np.uint64(1) << np.uint64(16)) | np.asarray(h, np.uint64)


def f16_normal(h):
    e = (np.asarray(h, np.uint32) >> 10) & 0x1F
    return (e >= 1) & (e <= 30)


def rtz_from_nearest(exact, near16):
    """binary16 toward zero from numpy's nearest binary16 of the same exact value."""
    beyond = np.abs(near16.astype(np.float64)) > np.abs(exact)
    return np.where(beyond, np.nextafter(near16, np.float16(0)), near16).view(np.uint16)


@pytest.mark.parametrize("op", ["mul", "add"])
def test_binary16_rtz_agreement(op):
    g = np.random.default_rng(21 if op == "mul" else 22)
    n = 1000000
    ha = g.integers(0, 1 << 16, n).astype(np.uint16)
    hb = g.integers(0, 1 << 16, n).astype(np.uint16)
    keep = f16_normal(ha) & f16_normal(hb)
    ha, hb = ha[keep], hb[keep]
    fa, fb = ha.view(np.float16).astype(np.float64), hb.view(np.float16).astype(np.float64)
    exact = fa * fb if op == "mul" else fa + fb
    with np.errstate(all="ignore"):
        near = exact.astype(np.float16)
    want = rtz_from_nearest(exact, near)
    # normal range of both, below binary16's overflow threshold (IEEE's toward-
    # zero overflow gives the largest finite value; this format gives infinity
    # only past the top binade, which the bound below excludes)
    keep = (np.abs(exact) >= 2.0 ** -14) & (np.abs(exact) < 65504.0) & f16_normal(want) & \
        (exact != 0)
    fn = orc.mul if op == "mul" else orc.add
    args = (5, 10, 10) if op == "mul" else (5, 10)
    got = fn(f16_code(ha[keep]), f16_code(hb[keep]), *args, rnd=RTZ)
    assert keep.sum() > 100000
    assert np.array_equal(got, f16_code(want[keep]))


def test_rtz_invariants():
    """|rtz(v)| <= |rne(v)| and |rtz(v)| <= |v|; rtz == rne when rne is exact;
    rtz is within one ulp of v."""
    g = np.random.default_rng(23)
    wE, wF, wFo = 5, 10, 11
    n = 400000
    a = (np.uint64(1) << np.uint64(16)) | g.integers(0, 1 << 16, n).astype(np.uint64)
    b = (np.uint64(1) << np.uint64(16)) | g.integers(0, 1 << 16, n).astype(np.uint64)
    exact = bf.to_float64(a, wE, wF) * bf.to_float64(b, wE, wF)
    z = bf.to_float64(orc.mul(a, b, wE, wF, wFo, rnd=RTZ), wE, wFo)
    r = bf.to_float64(orc.mul(a, b, wE, wF, wFo), wE, wFo)
    fin = np.isfinite(z) & np.isfinite(r) & (z != 0)
    assert fin.sum() > n // 2
    assert np.all(np.abs(z[fin]) <= np.abs(exact[fin]))
    assert np.all(np.abs(z[fin]) <= np.abs(r[fin]))
    assert np.all(np.sign(z[fin]) == np.sign(exact[fin]))
    same = fin & (r == exact)
    assert np.array_equal(z[same], r[same])
    ulp = np.ldexp(1.0, (np.floor(np.log2(np.abs(z[fin]))) - wFo).astype(np.int64))
    assert np.all(np.abs(exact[fin]) - np.abs(z[fin]) < ulp)


def test_rtz_conv_order_and_mode():
    """A conv in toward-zero mode equals the loop of toward-zero mul and add
    written out here; it differs from the nearest-even conv somewhere."""
    g = np.random.default_rng(24)
    ifm = g.integers(0, 1 << 11, (1, 4, 4, 5)).astype(np.uint64) | (np.uint64(1) << np.uint64(9))
    ifm &= np.uint64((1 << 10) - 1) | (np.uint64(1) << np.uint64(9))  # normal codes
    w = (g.integers(0, 1 << 9, (3, 3, 5, 3)).astype(np.uint64)) | (np.uint64(1) << np.uint64(9))
    got = orc.conv2d(ifm, w, 1, 1, 5, 3, 4, 3, rnd=RTZ)
    want = np.zeros_like(got)
    for oy in range(4):
        for ox in range(4):
            for m in range(3):
                acc = np.uint64(0)
                for ky in range(3):
                    for kx in range(3):
                        for c in range(5):
                            iy, ix = oy + ky - 1, ox + kx - 1
                            x = ifm[0, iy, ix, c] if 0 <= iy < 4 and 0 <= ix < 4 else np.uint64(0)
                            p = bf.mul(np.array([w[ky, kx, c, m]]), np.array([x]), 5, 3, 4, "rtz")
                            acc = bf.add(np.array([acc]), p, 5, 4, "rtz")[0]
                want[0, oy, ox, m] = bf.convert(np.array([acc]), 5, 4, 3, "rtz")[0]
    assert np.array_equal(got, want)
    assert not np.array_equal(got, orc.conv2d(ifm, w, 1, 1, 5, 3, 4, 3))
