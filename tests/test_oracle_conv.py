"""Pins for the oracle's MCMK convolution (paper Sec. 3.4), CPU only."""
import numpy as np
import pytest

import bruteforce as bf
import oracle as orc
from paper_2007_06563_amd import inputs as I

WE, WF, WACC = 5, 3, 4


def ref_conv(ifm, w, stride, pad, wE, wF_in, wF_acc, wF_out, act=0, mode="rne"):
    """Convolution written as the plain loop over (ky, kx, c) with the
    brute-force reference operations, vectorised over all outputs at once."""
    N, H, W, C = ifm.shape
    KH, KW, _, M = w.shape
    OH = (H + 2 * pad - KH) // stride + 1
    OW = (W + 2 * pad - KW) // stride + 1
    zero_in = np.uint64(0)
    padded = np.full((N, H + 2 * pad, W + 2 * pad, C), zero_in, np.uint64)
    padded[:, pad:pad + H, pad:pad + W, :] = ifm
    acc = np.zeros((N, OH, OW, M), np.uint64)  # +0
    for ky in range(KH):
        for kx in range(KW):
            for c in range(C):
                x = padded[:, ky:ky + stride * OH:stride, kx:kx + stride * OW:stride, c]
                x = np.broadcast_to(x[..., None], acc.shape)
                wv = np.broadcast_to(w[ky, kx, c, :], acc.shape)
                acc = bf.add(acc, bf.mul(wv, x, wE, wF_in, wF_acc, mode), wE, wF_acc, mode)
    if act:
        acc = bf.relu(acc, wE, wF_acc)
    return bf.convert(acc, wE, wF_acc, wF_out, mode)


def small_conv_codes():
    ifm, w = I.small_conv_inputs()
    return orc.quantize_f32(ifm, WE, WF), orc.quantize_f32(w, WE, WF)


def test_small_conv_matches_plain_loop():
    ifm, w = small_conv_codes()
    got = orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC)
    assert got.shape == (1, 8, 8, 8)
    assert np.array_equal(got, ref_conv(ifm, w, 1, 1, WE, WF, WACC, WACC))


@pytest.mark.parametrize("stride,pad,k", [(2, 1, 3), (2, 0, 1), (1, 0, 3), (3, 2, 3)])
def test_strides_and_padding_match_plain_loop(stride, pad, k):
    g = np.random.default_rng(stride * 10 + pad)
    ifm = orc.quantize_f32(g.uniform(-2, 2, (2, 7, 9, 5)).astype(np.float32), WE, WF)
    w = orc.quantize_f32(g.uniform(-1, 1, (k, k, 5, 6)).astype(np.float32), WE, WF)
    for act, wout in ((0, WACC), (1, 5), (1, 3)):
        got = orc.conv2d(ifm, w, stride, pad, WE, WF, WACC, wout, act=act)
        assert np.array_equal(got, ref_conv(ifm, w, stride, pad, WE, WF, WACC, wout, act)), (act, wout)


def test_special_values_in_conv_match_plain_loop():
    g = np.random.default_rng(77)
    ifm = orc.quantize_f32(I.inject_specials(g.uniform(-2, 2, (1, 5, 5, 3)).astype(np.float32),
                                             g, 0.1), WE, WF)
    w = orc.quantize_f32(I.inject_specials(g.uniform(-2, 2, (3, 3, 3, 4)).astype(np.float32),
                                           g, 0.05), WE, WF)
    got = orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC)
    assert np.array_equal(got, ref_conv(ifm, w, 1, 1, WE, WF, WACC, WACC))


def test_delta_kernel_returns_widened_ifm():
    ifm, _ = small_conv_codes()
    C = ifm.shape[-1]
    one = orc.quantize_f32(np.array([1.0], np.float32), WE, WF)[0]
    w = np.zeros((3, 3, C, C), np.uint64)
    for c in range(C):
        w[1, 1, c, c] = one
    got = orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC)
    widened = orc.convert(ifm, WE, WF, WACC)
    # -0 inputs come out as +0 (the accumulator starts at +0)
    widened[widened == np.uint64(1 << (WE + WACC))] = 0
    assert np.array_equal(got, widened)
    # and the values are the IFM's own
    assert np.array_equal(orc.decode_f32(got, WE, WACC), orc.decode_f32(ifm, WE, WF) + 0.0)


def test_zero_weights_give_positive_zero():
    ifm, w = small_conv_codes()
    got = orc.conv2d(ifm, np.zeros_like(w), 1, 1, WE, WF, WACC, WACC)
    assert np.all(got == 0)


def test_1x1_single_channel_is_one_multiply():
    ifm, w = small_conv_codes()
    x = ifm[..., :1]
    wv = w[1:2, 1:2, :1, :]
    got = orc.conv2d(x, wv, 1, 0, WE, WF, WACC, WACC)
    p = bf.mul(np.broadcast_to(wv[0, 0, 0], got.shape), np.broadcast_to(x, got.shape), WE, WF, WACC)
    assert np.array_equal(got, bf.add(np.zeros_like(p), p, WE, WACC))


def test_accumulation_order_matters():
    """Reversing the channel order changes some outputs, so the fixed order is
    observable (rounding after every add makes the sum order-dependent)."""
    g = np.random.default_rng(5)
    ifm = orc.quantize_f32(np.abs(g.standard_normal((1, 6, 6, 32))).astype(np.float32), WE, WF)
    w = orc.quantize_f32((g.standard_normal((3, 3, 32, 8)) * 0.3).astype(np.float32), WE, WF)
    a = orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC)
    b = orc.conv2d(ifm[..., ::-1].copy(), w[:, :, ::-1, :].copy(), 1, 1, WE, WF, WACC, WACC)
    assert np.any(a != b)


def test_points_match_full_and_threads_agree():
    ifm, w = small_conv_codes()
    full = orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC, nthreads=1)
    assert np.array_equal(full, orc.conv2d(ifm, w, 1, 1, WE, WF, WACC, WACC, nthreads=5))
    g = np.random.default_rng(0)
    pts = np.stack([np.zeros(50, int), g.integers(0, 8, 50), g.integers(0, 8, 50),
                    g.integers(0, 8, 50)], 1)
    got = orc.conv2d_points(ifm, w, pts, 1, 1, WE, WF, WACC, WACC)
    assert np.array_equal(got, full[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]])
