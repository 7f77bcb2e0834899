"""GPU parity of global average pooling (through the C ABI) against the oracle.

The pooling layer is the one the paper proposes for the interface between
MobileNets' last convolution and its fully connected layer (Sec. 4). Every
comparison is of codes: zero mismatches allowed. Inputs are seeded; each case
prints what it runs before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from gpu_util import dev, need_gpu, say
from paper_2007_06563_amd import inputs as I
from paper_2007_06563_amd import variants
from planes import pack_codes, unpack_planes

pytestmark = pytest.mark.gpu


def pool_inputs(seed, N, H, W, C, wE, wF, specials=0.0):
    """Codes of N(0,1) values in (wE, wF), NHWC, a share of them specials."""
    g = np.random.default_rng([11, seed])
    x = g.normal(size=N * H * W * C).astype(np.float32)
    if specials:
        x = I.inject_specials(x, g, specials)
    return orc.quantize_f32(x.reshape(N, H, W, C), wE, wF)


def run_pool(hf, codes, wE, wi, wa, wo, rnd):
    N, H, W, C = codes.shape
    planes = pack_codes(codes.reshape(N * H * W, C), 3 + wE + wi)
    out = hf.avgpool(dev(planes.view(np.int32)), N, H, W, C, (wE, wi), (wE, wa), (wE, wo),
                     round=rnd)
    torch.cuda.synchronize()
    return unpack_planes(out.cpu().numpy(), C)


@pytest.mark.parametrize("v", variants.POOL_VARIANTS, ids=variants.pool_tag)
def test_avgpool_every_variant(v):
    """A ragged channel count (40: one full word, one of 8) and a 3 x 5 map;
    2% of the inputs are zeros, infinities or NaNs."""
    hf = need_gpu()
    wE, wi, wa, wo, rnd = v
    x = pool_inputs(sum(v), 2, 3, 5, 40, wE, wi, specials=0.02)
    say(f"avgpool {variants.pool_tag(v)} shape={x.shape}")
    got = run_pool(hf, x, wE, wi, wa, wo, rnd)
    want = orc.avgpool(x, wE, wi, wa, wo, rnd=rnd)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("rnd", [variants.RNE, variants.RTZ], ids=["rne", "rtz"])
def test_avgpool_every_pair_of_codes(rnd):
    """Two positions per image and channel, (5,4) in and out: every pair of
    codes (x1, x2) -- 2^24 of them, non-canonical specials included -- as one
    (image, channel), so the adder sees every canonical accumulator value
    against every code, then the multiply by 1/2. Against the oracle."""
    hf = need_gpu()
    N, C = 1 << 12, 1 << 12
    i = np.arange(N * C, dtype=np.uint64)
    x = np.stack([i & np.uint64(C - 1), i >> np.uint64(12)], axis=1)  # [pair, position]
    codes = x.reshape(N, C, 2).transpose(0, 2, 1).reshape(N, 1, 2, C).copy()
    say(f"avgpool every pair of (5,4) codes rnd={rnd}")
    got = run_pool(hf, codes, 5, 4, 4, 4, rnd)
    want = orc.avgpool(codes, 5, 4, 4, 4, rnd=rnd)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches; first at {bad[0]}"


@pytest.mark.parametrize("rnd", [variants.RNE, variants.RTZ], ids=["rne", "rtz"])
def test_avgpool_mobilenet_interface(rnd):
    """The MobileNets shape: batch 16, the last 7 x 7 x 1024 feature map, (5,4)."""
    hf = need_gpu()
    x = pool_inputs(5, 16, 7, 7, 1024, 5, 4)
    say(f"avgpool mobilenet 16x7x7x1024 (5,4) round={rnd}")
    got = run_pool(hf, x, 5, 4, 4, 4, rnd)
    assert np.array_equal(got, orc.avgpool(x, 5, 4, 4, 4, rnd=rnd))


@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (3, 1, 1, 33), (1, 56, 56, 64), (5, 2, 9, 31)],
                         ids=lambda s: "x".join(map(str, s)))
def test_avgpool_edge_shapes(shape):
    """One position (a multiply by one), one channel, a 3136-position map (the
    scale 1/3136), a count of channels below one word."""
    hf = need_gpu()
    x = pool_inputs(len(shape) + shape[3], *shape, 5, 4, specials=0.01)
    say(f"avgpool edge shape={shape}")
    got = run_pool(hf, x, 5, 4, 5, 4, variants.RNE)
    assert np.array_equal(got, orc.avgpool(x, 5, 4, 5, 4))


def test_avgpool_of_a_conv_output():
    """Conv (planes stay on the GPU) then pooling, as at the end of a network."""
    hf = need_gpu()
    g = np.random.default_rng(9)
    ifm = g.normal(size=(2, 9, 9, 32)).astype(np.float32)
    w = (g.normal(size=(3, 3, 32, 48)) * 0.1).astype(np.float32)
    say("conv 2x9x9x32 -> 48 then avgpool (5,4)")
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    pi = hf.pack(dev(ifm.reshape(-1, 32)), (5, 3))
    pw = hf.pack(dev(w.reshape(-1, 48)), (5, 3))
    d = hf.conv_desc(2, 9, 9, 32, 48, 3, 3, 1, 1, (5, 3), (5, 4), (5, 4), 0)
    o = hf.conv2d(pi, pw, d)
    pooled = hf.avgpool(o, 2, 9, 9, 48, (5, 4), (5, 4), (5, 4))
    torch.cuda.synchronize()
    got = unpack_planes(pooled.cpu().numpy(), 48)
    ref = orc.conv2d(qi, qw, 1, 1, 5, 3, 4, 4)
    assert np.array_equal(got, orc.avgpool(ref, 5, 4, 4, 4))
