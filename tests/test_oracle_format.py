"""Pins for the oracle's number format, quantizer and decoder (CPU only)."""
import json
import os

import numpy as np
import pytest
import torch

import bruteforce as bf
import oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_mac_type_widths_match_table3():
    """NINBITS = 2 + 1 + wE + wF and the single/extended output widths
    (paper Table 3 and the HOBFLOPS9 example of Sec. 3.4)."""
    g = json.load(open(os.path.join(GOLDEN, "mac_types.json")))
    for t in g["types"]:
        wE, wF = t["in"]
        assert t["out_single"] == [wE, wF + 1]
        assert t["out_extended"] == [wE, 2 * wF + 1]
    h = g["hobflops9_bits"]
    wE, wF = 5, 3
    assert 3 + wE + wF == h["NINBITS"]
    assert 3 + wE + wF + 1 == h["NOUTBITS_single"]
    assert 3 + wE + 2 * wF + 1 == h["NOUTBITS_extended"]
    # and the oracle handles all of those formats: widening the largest input
    # value of each type to the output types is exact
    for t in g["types"]:
        wE, wF = t["in"]
        top = (1 << (wF + wE + 1)) | (((1 << wE) - 1) << wF) | ((1 << wF) - 1)
        for wFo in (t["out_single"][1], t["out_extended"][1]):
            r = int(orc.convert(np.array([top], np.uint64), wE, wF, wFo)[0])
            assert r == (1 << (wFo + wE + 1)) | (((1 << wE) - 1) << wFo) | \
                (((1 << wF) - 1) << (wFo - wF))


def test_hand_worked_examples():
    g = json.load(open(os.path.join(GOLDEN, "hand_examples.json")))
    for c in g["cases"]:
        want = int(c["code"], 16)
        if c["op"] == "quantize":
            got = orc.quantize_f32(np.array([c["x"]], np.float32), *c["fmt"])[0]
        elif c["op"] == "mul":
            wE, wF = c["fmt_in"]
            got = orc.mul(np.array([int(c["a"], 16)], np.uint64),
                          np.array([int(c["b"], 16)], np.uint64), wE, wF, c["wF_out"])[0]
        else:
            got = orc.add(np.array([int(c["a"], 16)], np.uint64),
                          np.array([int(c["b"], 16)], np.uint64), *c["fmt"])[0]
        assert int(got) == want, c


@pytest.mark.parametrize("wE,wF", [(4, 2), (5, 3), (5, 4), (5, 10), (5, 11), (8, 7), (8, 8)])
def test_decode_quantize_round_trip(wE, wF):
    """Every normal code decodes to a float32 that quantizes back to itself;
    special codes with arbitrary fields come back canonical."""
    c = np.arange(1 << (3 + wE + wF), dtype=np.uint64)
    f = orc.decode_f32(c, wE, wF)
    back = orc.quantize_f32(f, wE, wF)
    exn = (c >> np.uint64(wE + wF + 1)) & np.uint64(3)
    sbit = (c >> np.uint64(wE + wF)) & np.uint64(1)
    Ebits = (c >> np.uint64(wF)) & np.uint64((1 << wE) - 1)
    in_f32 = np.ones(c.shape, bool)
    if wE == 8:  # E = 0 and E = 255 lie outside float32's normal range
        in_f32 = (Ebits >= 1) & (Ebits <= 254)
    normal = (exn == 1) & in_f32
    assert np.array_equal(back[normal], c[normal])
    es = np.uint64(wE + wF + 1)
    canon = np.where(exn == 3, np.uint64(3) << es,
                     (exn << es) | (sbit << np.uint64(wE + wF)))
    sp = exn != 1
    assert np.array_equal(back[sp], canon[sp])


def test_decode_agrees_with_ieee_bit_patterns():
    """Normal (5,10), (8,7) and (8,23) codes carry the binary16, bfloat16 and
    binary32 sign/exponent/fraction fields unchanged."""
    h = np.arange(1 << 16, dtype=np.uint64)
    e = (h >> np.uint64(10)) & np.uint64(31)
    n = (e >= 1) & (e <= 30)
    got = orc.decode_f32(h[n] | np.uint64(1 << 16), 5, 10)
    want = h[n].astype(np.uint16).view(np.float16).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    e = (h >> np.uint64(7)) & np.uint64(255)
    n = (e >= 1) & (e <= 254)
    got = orc.decode_f32(h[n] | np.uint64(1 << 16), 8, 7)
    want = torch.from_numpy(h[n].astype(np.uint16).astype(np.int16)).view(torch.bfloat16).float()
    assert np.array_equal(got.view(np.uint32), want.numpy().view(np.uint32))
    g = np.random.default_rng(0)
    b = g.integers(0, 1 << 32, 1 << 20, dtype=np.uint64)
    e = (b >> np.uint64(23)) & np.uint64(255)
    b = b[(e >= 1) & (e <= 254)]
    got = orc.decode_f32(b | np.uint64(1 << 32), 8, 23)
    assert np.array_equal(got.view(np.uint32), b.astype(np.uint32))


def f16_ties_and_neighbours():
    """float32 values at and around every rounding boundary of binary16 normals."""
    h = np.arange(0x0400, 0x7C00, dtype=np.uint16)  # positive normals
    v = h.view(np.float16).astype(np.float32)
    nxt = (h + 1).view(np.float16).astype(np.float32)
    mid = ((v.astype(np.float64) + nxt.astype(np.float64)) / 2).astype(np.float32)  # exact
    u = mid.view(np.uint32)
    cand = np.concatenate([v, mid, (u + 1).view(np.float32), (u - 1).view(np.float32)])
    return np.concatenate([cand, -cand])


def test_quantize_matches_binary16_conversion():
    g = np.random.default_rng(12)
    r = g.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32).view(np.float32)
    x = np.concatenate([f16_ties_and_neighbours(), r])
    with np.errstate(all="ignore"):
        h = x.astype(np.float16).view(np.uint16)
    e = (h >> 10) & 31
    keep = (e >= 1) & (e <= 30) & (np.abs(x.astype(np.float64)) >= 2.0 ** -14)
    got = orc.quantize_f32(x[keep], 5, 10)
    assert keep.sum() > 200000
    assert np.array_equal(got, (np.uint64(1) << np.uint64(16)) | h[keep].astype(np.uint64))


def test_quantize_matches_bfloat16_conversion():
    g = np.random.default_rng(13)
    b = g.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32)
    # plus exact ties: bfloat16 pattern followed by 1000...0 in the dropped bits
    t = (g.integers(0, 1 << 16, 1 << 16).astype(np.uint32) << 16) | 0x8000
    x = np.concatenate([b, t]).view(np.float32)
    bf16 = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    e = (bf16 >> 7) & 255
    keep = (e >= 1) & (e <= 254) & np.isfinite(x) & (np.abs(x.astype(np.float64)) >= 2.0 ** -126)
    got = orc.quantize_f32(x[keep], 8, 7)
    assert np.array_equal(got, (np.uint64(1) << np.uint64(16)) | bf16[keep].astype(np.uint64))


@pytest.mark.parametrize("wE,wF", [(4, 2), (5, 2), (5, 3), (5, 5), (5, 7), (5, 10), (4, 3),
                                   (8, 7), (8, 10)])
def test_quantize_vs_bruteforce(wE, wF):
    g = np.random.default_rng(100 + wF)
    b = g.integers(0, 1 << 32, 1 << 19, dtype=np.uint64).astype(np.uint32)
    x = b.view(np.float32)
    x = np.concatenate([x, g.uniform(-4, 4, 1 << 18).astype(np.float32),
                        np.array([0.0, -0.0, np.inf, -np.inf, np.nan], np.float32)])
    assert np.array_equal(orc.quantize_f32(x, wE, wF), bf.quantize(x, wE, wF))


def test_quantize_f32_subnormals_exact():
    """(8,23) has normal binades below float32's; float32 subnormals with at most
    23 significant bits land there exactly (E = 0 covers [2^-127, 2^-126))."""
    sub = np.array([0x00400000, 0x00600000, 0x007FFFFF], np.uint32).view(np.float32)
    got = orc.quantize_f32(sub, 8, 23)
    back = bf.to_float64(got, 8, 23)
    assert np.array_equal(back, sub.astype(np.float64))
