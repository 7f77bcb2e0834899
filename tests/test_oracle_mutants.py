"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of the oracle's C source, compiles it
and runs a reduced set of the pins on it; every mutant must fail at least one.
The unmodified source must pass the same set, so the check itself is sound.
"""
import os
import subprocess

import numpy as np
import pytest

import bruteforce as bf
import oracle as orc
from oracle import build as obuild
from test_oracle_conv import ref_conv
from test_oracle_pool import nearest_rational

SRC = open(obuild.SRC).read()

MUTANTS = {
    "ties_away": ("int round_up = mode == HFO_RNE && half_bit && (below_half || (sig & 1));",
                  "int round_up = mode == HFO_RNE && half_bit;"),
    "truncate": ("int round_up = mode == HFO_RNE && half_bit && (below_half || (sig & 1));",
                 "int round_up = 0;"),
    "rtz_rounds_to_nearest": ("int round_up = mode == HFO_RNE && half_bit && (below_half || (sig & 1));",
                              "int round_up = half_bit && (below_half || (sig & 1));"),
    "rtz_rounds_up": ("int round_up = mode == HFO_RNE && half_bit && (below_half || (sig & 1));",
                      "int round_up = mode == HFO_RNE ? half_bit && (below_half || (sig & 1)) : (half_bit || below_half);"),
    "conv_ignores_mode": ("acc = hfo_add_rm(acc, p, d->wE, d->wF_acc, d->round);",
                          "acc = hfo_add_rm(acc, p, d->wE, d->wF_acc, HFO_RNE);"),
    "sticky_dropped": ("int below_half = big_any_below(M, k - 1);", "int below_half = 0;"),
    "no_renormalise": ("sig >>= 1;\n      u += 1;", "sig >>= 1;"),
    "bias_off_by_one": ("return ((int64_t)1 << (f.wE - 1)) - 1;", "return ((int64_t)1 << (f.wE - 1));"),
    "E0_reserved": ("if (Eb < 0) return make_zero(s, f);", "if (Eb < 1) return make_zero(s, f);"),
    "Emax_reserved": ("if (Eb > (((int64_t)1 << f.wE) - 1)) return make_inf(s, f);",
                      "if (Eb >= (((int64_t)1 << f.wE) - 1)) return make_inf(s, f);"),
    "cancel_sign": ("if (c == 0) return make_zero(0, f);", "if (c == 0) return make_zero(A.s, f);"),
    "zero_zero_sign": ("make_zero(A.s & B.s, f)", "make_zero(A.s | B.s, f)"),
    "zero_times_inf": ("if ((A.exn == EXN_INF && B.exn == EXN_ZERO) || (A.exn == EXN_ZERO && B.exn == EXN_INF))",
                       "if (0)"),
    "inf_minus_inf": ("return A.s == B.s ? make_inf(A.s, f) : make_nan(f);", "return make_inf(A.s, f);"),
    "sub_sign": ("      s = B.s;", "      s = A.s;"),
    "product_exponent": ("exp2_of(A, fi) + exp2_of(B, fi), mode);",
                         "exp2_of(A, fi) + exp2_of(B, fi) + 1, mode);"),
    "align_wrong_operand": ("big_set_shl(&Y, sig_of(B, f), (int)(eb - emin));",
                            "big_set_shl(&Y, sig_of(B, f), (int)(ea - emin));"),
    "relu_keeps_neg_zero": ("if (A.s) return make_zero(0, f);",
                            "if (A.s && A.exn != EXN_ZERO) return make_zero(0, f);"),
    "nan_sign": ("static uint64_t make_nan(fmt_t f) { return encode(EXN_NAN, 0, 0, 0, f); }",
                 "static uint64_t make_nan(fmt_t f) { return encode(EXN_NAN, 1, 0, 0, f); }"),
    "subnormal_scale": ("int64_t e = ef ? (int64_t)ef - 150 : -149;", "int64_t e = ef ? (int64_t)ef - 150 : -150;"),
    "channel_order": ("for (int c = 0; c < d->C; c++) {", "for (int c = d->C - 1; c >= 0; c--) {"),
    "padding_index": ("int ix = ox * d->stride + kx - d->pad;", "int ix = ox * d->stride + kx;"),
    "relu_after_convert": ("  if (d->act == 1) acc = hfo_relu(acc, d->wE, d->wF_acc);\n  return hfo_convert_rm(",
                           "  return hfo_convert_rm("),
    "pool_columns_first": ("for (int y = 0; y < H; y++) {\n        for (int x = 0; x < W; x++) {",
                           "for (int x = 0; x < W; x++) {\n        for (int y = 0; y < H; y++) {"),
    "pool_starts_at_neg_zero": ("uint64_t acc = make_zero(0, fa);", "uint64_t acc = make_zero(1, fa);"),
    "pool_ignores_mode": ("acc = hfo_add_rm(acc, hfo_convert_rm(v, wE, wF_in, wF_acc, round), wE, wF_acc, round);",
                          "acc = hfo_add_rm(acc, hfo_convert_rm(v, wE, wF_in, wF_acc, round), wE, wF_acc, HFO_RNE);"),
    "recip_truncated": ("return round_value(f, 0, &M, -(int64_t)k - 1, HFO_RNE);",
                        "return round_value(f, 0, &M, -(int64_t)k - 1, HFO_RTZ);"),
    "recip_no_sticky": ("big_set_shl(&M, (q << 1) | (r != 0), 0);", "big_set_shl(&M, q << 1, 0);"),
    "pool_scale_missing": ("out[(size_t)n * C + c] = hfo_mul_rm(acc, scale, wE, wF_acc, wF_out, round);",
                           "out[(size_t)n * C + c] = hfo_convert_rm(acc, wE, wF_acc, wF_out, round);"),
}


def compile_variant(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    c.write_text(src)
    so = tmp_path / f"{name}.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-pthread", "-I",
                    os.path.dirname(obuild.SRC), "-o", str(so), str(c), "-lm"], check=True)
    return orc.load(str(so))


@pytest.fixture(scope="module")
def refs():
    r = {}
    n = 1 << 11
    a = np.repeat(np.arange(n, dtype=np.uint64), n)
    b = np.tile(np.arange(n, dtype=np.uint64), n)
    r["mul"] = (a, b, bf.mul(a, b, 5, 3, 4))
    n = 1 << 10
    a2 = np.repeat(np.arange(n, dtype=np.uint64), n)
    b2 = np.tile(np.arange(n, dtype=np.uint64), n)
    r["add"] = (a2, b2, bf.add(a2, b2, 4, 3))
    cv = np.arange(1 << 12, dtype=np.uint64)
    r["relu"] = (cv, bf.relu(cv, 5, 4))
    g = np.random.default_rng(3)
    x = np.concatenate([g.integers(0, 1 << 32, 1 << 16, dtype=np.uint64).astype(np.uint32).view(np.float32),
                        np.array([1e-40, 3e-39, -2e-39], np.float32)])
    r["q"] = (x, bf.quantize(x, 5, 3), bf.quantize(x, 8, 7))
    ifm = bf.quantize(g.uniform(-2, 2, (1, 5, 6, 4)).astype(np.float32), 5, 3)
    w = bf.quantize(g.uniform(-1, 1, (3, 3, 4, 3)).astype(np.float32), 5, 3)
    r["conv"] = (ifm, w, ref_conv(ifm, w, 1, 1, 5, 3, 4, 4), ref_conv(ifm, w, 1, 1, 5, 3, 4, 4, act=1))
    r["mul_rtz"] = bf.mul(a, b, 5, 3, 4, mode="rtz")
    r["add_rtz"] = bf.add(a2, b2, 4, 3, mode="rtz")
    r["conv_rtz"] = ref_conv(ifm, w, 1, 1, 5, 3, 4, 3, mode="rtz")
    # pooling: the nearest codes of 1/n, and a 4 x 4 map whose mean depends on
    # the summation order (see test_oracle_pool)
    from fractions import Fraction
    r["recip"] = [(n, nearest_rational(Fraction(1, n), 5, 10)) for n in range(1, 200)]
    maps = np.ones((3, 4, 4, 1), np.float32)
    maps[0, 3, 3, 0] = maps[1, 0, 0, 0] = maps[2, 0, 3, 0] = 64.0
    r["pool_order"] = (bf.quantize(maps, 5, 3), bf.quantize(np.array([[5.0], [4.0], [4.0]], np.float32), 5, 3))
    r["pool_zero"] = (bf.quantize(np.full((1, 2, 2, 1), -0.0, np.float32), 5, 4), np.zeros((1, 1), np.uint64))
    pos = np.abs(g.normal(size=(1, 7, 7, 16))).astype(np.float32) + 0.01
    xp = bf.quantize(pos, 5, 4)
    scale = np.full(16, nearest_rational(Fraction(1, 49), 5, 4), np.uint64)
    acc = np.zeros(16, np.uint64)
    for i in range(49):               # rows, then columns; truncating adds
        acc = bf.add(acc, xp.reshape(49, 16)[i], 5, 4, mode="rtz")
    r["pool_rtz"] = (xp, bf.mul(acc, scale, 5, 4, 4, mode="rtz").reshape(1, 16))
    return r


def failures(L, r):
    """Names of the reduced pins that library L fails."""
    bad = []
    a, b, want = r["mul"]
    if not np.array_equal(orc.mul(a, b, 5, 3, 4, L=L), want):
        bad.append("mul")
    a, b, want = r["add"]
    if not np.array_equal(orc.add(a, b, 4, 3, L=L), want):
        bad.append("add")
    cv, want = r["relu"]
    if not np.array_equal(orc.relu(cv, 5, 4, L=L), want):
        bad.append("relu")
    x, q53, q87 = r["q"]
    if not (np.array_equal(orc.quantize_f32(x, 5, 3, L=L), q53)
            and np.array_equal(orc.quantize_f32(x, 8, 7, L=L), q87)):
        bad.append("quantize")
    ifm, w, want, want_relu = r["conv"]
    if not np.array_equal(orc.conv2d(ifm, w, 1, 1, 5, 3, 4, 4, L=L), want):
        bad.append("conv")
    if not np.array_equal(orc.conv2d(ifm, w, 1, 1, 5, 3, 4, 4, act=1, L=L), want_relu):
        bad.append("conv_relu")
    a, b, _ = r["mul"]
    if not np.array_equal(orc.mul(a, b, 5, 3, 4, L=L, rnd=orc.RTZ), r["mul_rtz"]):
        bad.append("mul_rtz")
    a, b, _ = r["add"]
    if not np.array_equal(orc.add(a, b, 4, 3, L=L, rnd=orc.RTZ), r["add_rtz"]):
        bad.append("add_rtz")
    if not np.array_equal(orc.conv2d(ifm, w, 1, 1, 5, 3, 4, 3, L=L, rnd=orc.RTZ), r["conv_rtz"]):
        bad.append("conv_rtz")
    if any(int(orc.recip(n, 5, 10, L=L)) != want for n, want in r["recip"]):
        bad.append("recip")
    maps, want = r["pool_order"]
    if not np.array_equal(orc.avgpool(maps, 5, 3, 3, 3, L=L), want):
        bad.append("pool_order")
    zeros, want = r["pool_zero"]
    if not np.array_equal(orc.avgpool(zeros, 5, 4, 4, 4, L=L), want):
        bad.append("pool_zero")
    x, want = r["pool_rtz"]
    if not np.array_equal(orc.avgpool(x, 5, 4, 4, 4, L=L, rnd=orc.RTZ), want):
        bad.append("pool_rtz")
    return bad


def test_unmodified_oracle_passes_reduced_pins(tmp_path, refs):
    assert failures(compile_variant(tmp_path, "orig", SRC), refs) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, refs, name):
    old, new = MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation site for {name} not unique"
    L = compile_variant(tmp_path, name, SRC.replace(old, new))
    assert failures(L, refs), f"mutant {name} passed every pin"
