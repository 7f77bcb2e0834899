"""GPU parity at the workloads' full sizes.

Each workload runs whole on the GPU through the C ABI, at its real shape:
  * the small convolution 8x8x4 -> 8 accumulating in its own input format
    (5,3), as well as in (5,4): every output;
  * the element-wise a*b+c sweep: 2^24 triples per format, six formats: every
    triple;
  * the ResNet layer 8x56x56x64 -> 64 in the benchmark's launch (split kernel,
    float32 OFM written by the epilogue): every output;
  * the paper's MobileNets-shaped layer 14x14x512 -> 512, 3x3, stride 2, for
    every generated MAC type of the type sweep: every output;
  * the mantissa sweep: 4x224x224x3 -> 64 and 4x28x28x256 -> 512, 3x3, for
    input formats (5, m), m = 2..10, accumulating in (5, m+1): a sample;
  * the 13-layer stack's first layer in all four kernel shapes: every output
    equal across them, a sample against the oracle;
  * the 13-layer ResNet-shaped stack at batch 16, planes kept on the GPU from
    layer to layer, ReLU and a format change in every epilogue: a sample.
Where the oracle recomputes a sample, it takes every border position of every
image plus random points, and the codes must agree bit for bit. For the stack
the oracle's input to each layer is the GPU's own output of the previous layer
(teacher forcing), so every layer is checked on its own; the first layer's
input and all weights are quantised by the oracle.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as orc
from gpu_util import codes_of, dev, need_gpu, say
from paper_2007_06563_amd import inputs as I

pytestmark = pytest.mark.gpu

SAMPLES = 65536


def threaded(fn, *arrays, fixed=()):
    """An element-wise oracle function over chunks of equally shaped arrays,
    one chunk per host thread (the oracle itself is unchanged)."""
    n = arrays[0].size
    t = max(1, min(orc.default_threads(), 16))
    bounds = np.linspace(0, n, t + 1).astype(np.int64)
    flat = [a.reshape(-1) for a in arrays]
    with ThreadPoolExecutor(t) as ex:
        parts = list(ex.map(lambda i: fn(*[a[bounds[i]:bounds[i + 1]] for a in flat], *fixed),
                            range(t)))
    return np.concatenate(parts).reshape(arrays[0].shape)


@pytest.mark.parametrize("idx", range(len(I.FMA_FORMATS)),
                         ids=[f"e{e}m{m}" for e, m in I.FMA_FORMATS])
def test_fma_sweep_every_triple(idx):
    """2^24 triples, U[-4,4] with 1 % specials per operand: all computed on the
    GPU (pack, muladd, unpack to codes and to float32) and all recomputed by
    the oracle."""
    hf = need_gpu()
    wE, wF = I.FMA_FORMATS[idx]
    wa = wF + 1
    a, b, c = I.fma_operands(idx)
    n = a.size
    say(f"fma sweep ({wE},{wF}) -> ({wE},{wa}) n={n}")
    pa, pb, pc = (hf.pack(dev(t.reshape(1, n)), (wE, wF)) for t in (a, b, c))
    r = hf.muladd(pa, pb, pc, n, (wE, wF), (wE, wa))
    got = codes_of(hf.unpack(r, 1, n, (wE, wa), kind="code"))[0]
    got_f = hf.unpack(r, 1, n, (wE, wa), kind="f32").cpu().numpy().view(np.uint32)[0]
    qa, qb, qc = (threaded(orc.quantize_f32, t, fixed=(wE, wF)) for t in (a, b, c))
    want = threaded(orc.muladd, qa, qb, qc, fixed=(wE, wF, wa))
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches of {n}; first at {bad[0]}"
    want_f = threaded(orc.decode_f32, want, fixed=(wE, wa)).view(np.uint32)
    assert np.array_equal(got_f, want_f)


@pytest.mark.parametrize("algo", [1, 2], ids=["fused", "split"])
@pytest.mark.parametrize("rnd", [0, 1], ids=["rne", "rtz"])
@pytest.mark.parametrize("wa", [3, 4], ids=["acc_e5m3", "acc_e5m4"])
def test_small_conv_every_output(wa, rnd, algo):
    """The 8x8x4 -> 8 convolution, (5,3) inputs, accumulating in the same
    format (5,3) as the workload states it literally, and in (5,4), the
    paper's single MAC type: every output against the oracle."""
    hf = need_gpu()
    ifm, w = I.small_conv_inputs()
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    say(f"small conv acc=(5,{wa}) rnd={rnd} algo={algo}")
    got = conv_codes_of(hf, qi, qw, 1, 1, 5, 3, wa, wa, 0, algo, rnd)
    want = orc.conv2d(qi, qw, 1, 1, 5, 3, wa, wa, rnd=rnd)
    assert np.array_equal(got, want)


def conv_codes_of(hf, qi, qw, stride, pad, wE, wi, wa, wo, act, algo, rnd):
    """GPU convolution of code tensors (NHWC / HWIO) -> output codes."""
    N, H, W, C = qi.shape
    KH, KW, _, M = qw.shape
    d = hf.conv_desc(N, H, W, C, M, KH, KW, stride, pad, (wE, wi), (wE, wa), (wE, wo), act,
                     algo, round=rnd)
    OH, OW = hf.conv_out_hw(d)
    pi = hf.pack(dev(qi.astype(np.uint32).view(np.int32).reshape(N * H * W, C)), (wE, wi))
    pw = hf.pack(dev(qw.astype(np.uint32).view(np.int32).reshape(KH * KW * C, M)), (wE, wi))
    out = hf.unpack(hf.conv2d(pi, pw, d), N * OH * OW, M, (wE, wo), kind="code")
    return codes_of(out).reshape(N, OH, OW, M)


def test_resnet_layer_every_output():
    """8x56x56x64 -> 64, 3x3, (5,3) -> (5,4), in the benchmark's launch: one
    pack launch for the IFM and the weights, the split kernel, float32 OFM
    from the epilogue. Every output's float32 bits and code against the
    oracle's full convolution (all host threads)."""
    hf = need_gpu()
    s = I.RESNET_CONV_SHAPE
    ifm, w = I.resnet_conv_inputs()
    P = s.N * s.OH * s.OW
    say("resnet layer 8x56x56x64->64 every output (split kernel, float32 OFM)")
    x_ifm, x_w = dev(ifm.reshape(-1, s.C)), dev(w.reshape(-1, s.M))
    pi, pw = hf.pack_batch([x_ifm, x_w], (5, 3))
    vals = {}
    for kind in (hf.OFM_F32, hf.OFM_CODE):
        d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, 3), (5, 4),
                         (5, 4), hf.ACT_NONE, hf.ALGO_SPLIT, ofm_kind=kind)
        vals[kind] = hf.conv2d(pi, pw, d).cpu().numpy().view(np.uint32)
    qi = threaded(orc.quantize_f32, ifm, fixed=(5, 3))
    qw = orc.quantize_f32(w, 5, 3)
    want = orc.conv2d(qi, qw, s.stride, s.pad, 5, 3, 4, 4).reshape(P, s.M)
    bad = np.argwhere(vals[hf.OFM_CODE].astype(np.uint64) != want)
    assert bad.size == 0, f"{len(bad)} mismatching codes of {want.size}; first at {bad[0]}"
    want_f = threaded(orc.decode_f32, want, fixed=(5, 4)).view(np.uint32)
    assert np.array_equal(vals[hf.OFM_F32], want_f)


def test_stack_layer_one_every_kernel_shape():
    """The 13-layer stack's first layer (16x56x56x64 -> 64, 3x3, (5,3) ->
    (5,4) -> (5,5) ReLU: 1,568 chain waves, between one and two per SIMD, so
    AUTO runs the compact split kernel): the four kernel shapes give the same
    codes at every output, and those codes match the oracle on every border
    position plus random points."""
    hf = need_gpu()
    s = I.resnet_stack_shapes(16)[0]
    ifm, w = I.conv_inputs(I.RESNET_STACK, 0, s)
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, 3), (5, 4), (5, 5),
                     1, hf.ALGO_AUTO)
    assert hf.conv2d_algo(d) == hf.ALGO_SPLIT_COMPACT
    outs = {}
    for algo in (hf.ALGO_AUTO, hf.ALGO_FUSED, hf.ALGO_SPLIT, hf.ALGO_SPLIT_COMPACT):
        say(f"stack layer 1 16x56x56x64->64 algo={algo}")
        outs[algo] = conv_codes_of(hf, qi, qw, s.stride, s.pad, 5, 3, 4, 5, 1, algo, 0)
    for algo, o in outs.items():
        assert np.array_equal(o, outs[hf.ALGO_AUTO]), f"algo {algo} differs from AUTO"
    pts = sample_points((s.N, s.OH, s.OW), s.M, np.random.default_rng(41), 8192)
    want = orc.conv2d_points(qi, qw, pts, s.stride, s.pad, 5, 3, 4, 5, 1)
    got = outs[hf.ALGO_AUTO][pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]]
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches; first at {pts[bad[0]]}"


def _type_sweep_variants():
    from paper_2007_06563_amd import variants as V
    names = {(4, 3): "HOBFLOPSIEEE8"}
    names.update({(5, m): f"HOBFLOPS{m + 6}" for m in range(2, 11)})
    out = []
    for wE, wi, wa, wo, act, rnd in V.CONV_VARIANTS:
        if act or (wE, wi) not in names or wa == wi:
            continue
        ext = wa == 2 * wi + 1
        out.append(pytest.param((wE, wi, wa, rnd),
                                id=names[(wE, wi)] + ("e" if ext else "") + V._sfx(rnd)))
    return out


@pytest.mark.parametrize("t", _type_sweep_variants())
def test_mobilenet_layer_every_output(t):
    """The paper's type sweep layer (14x14x512 -> 512, 3x3, stride 2, pad 1,
    batch 1: 25,088 outputs of 4,608 taps each) for every generated MAC type,
    single and extended, both roundings, in the launch the library picks
    (the split kernel): every output against the oracle."""
    hf = need_gpu()
    wE, wi, wa, rnd = t
    s = I.mobilenet_layer(1)
    ifm, w = I.type_sweep_inputs(1)
    say(f"mobilenet layer type ({wE},{wi})->({wE},{wa}) rnd={rnd}")
    qi, qw = orc.quantize_f32(ifm, wE, wi), orc.quantize_f32(w, wE, wi)
    got = conv_codes_of(hf, qi, qw, s.stride, s.pad, wE, wi, wa, wa, 0, hf.ALGO_AUTO, rnd)
    pts = np.stack(np.meshgrid(np.arange(s.N), np.arange(s.OH), np.arange(s.OW), np.arange(s.M),
                               indexing="ij"), -1).reshape(-1, 4).astype(np.int64)
    want = orc.conv2d_points(qi, qw, pts, s.stride, s.pad, wE, wi, wa, wa, rnd=rnd)
    bad = np.flatnonzero(got.reshape(-1) != want)
    assert bad.size == 0, f"{bad.size} mismatches of {want.size}; first at {pts[bad[0]]}"


def sample_points(shape_out, M, g, count):
    """Every border position of every image (random kernel) plus random points."""
    N, OH, OW = shape_out
    pts = []
    for n in range(N):
        for t in range(OW):
            pts += [(n, 0, t), (n, OH - 1, t)]
        for t in range(OH):
            pts += [(n, t, 0), (n, t, OW - 1)]
    pts = np.array(pts, np.int64)
    pts = np.concatenate([pts, g.integers(0, M, (len(pts), 1))], 1)
    rnd = np.stack([g.integers(0, N, count), g.integers(0, OH, count), g.integers(0, OW, count),
                    g.integers(0, M, count)], 1).astype(np.int64)
    return np.concatenate([pts, rnd])


def conv_codes(hf, planes, d, wo):
    OH, OW = hf.conv_out_hw(d)
    return codes_of(hf.unpack(planes, d.N * OH * OW, d.M, (5, wo), kind="code")).reshape(
        d.N, OH, OW, d.M)


@pytest.mark.parametrize("si", [0, 1], ids=["4x224x224x3-64", "4x28x28x256-512"])
@pytest.mark.parametrize("m", I.MANTISSA_SWEEP_WF)
def test_mantissa_sweep_sampled(m, si):
    hf = need_gpu()
    s = I.MANTISSA_SWEEP_SHAPES[si]
    ifm, w = I.mantissa_sweep_inputs(si, m)
    say(f"mantissa sweep m={m} shape={s}")
    d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, m), (5, m + 1),
                     (5, m + 1))
    pi = hf.pack(dev(ifm.reshape(-1, s.C)), (5, m))
    pw = hf.pack(dev(w.reshape(-1, s.M)), (5, m))
    got = conv_codes(hf, hf.conv2d(pi, pw, d), d, m + 1)
    qi = threaded(orc.quantize_f32, ifm, fixed=(5, m))
    qw = orc.quantize_f32(w, 5, m)
    pts = sample_points((s.N, s.OH, s.OW), s.M, np.random.default_rng([2, si, m]), SAMPLES)
    want = orc.conv2d_points(qi, qw, pts, s.stride, s.pad, 5, m, m + 1, m + 1)
    bad = np.flatnonzero(got[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]] != want)
    assert bad.size == 0, f"{bad.size} mismatches of {len(pts)}; first at {pts[bad[0]]}"


def test_resnet_stack_teacher_forced():
    """The 13 layers at batch 16; planes never leave the GPU between layers."""
    hf = need_gpu()
    shapes = I.resnet_stack_shapes(16)
    fmts = I.resnet_stack_formats(len(shapes))
    ifm0, _ = I.conv_inputs(I.RESNET_STACK, 0, shapes[0])
    planes = hf.pack(dev(ifm0.reshape(-1, shapes[0].C)), (5, fmts[0][0]))
    in_codes = threaded(orc.quantize_f32, ifm0, fixed=(5, fmts[0][0]))
    for li, (s, (wi, wa, wo)) in enumerate(zip(shapes, fmts)):
        _, w = I.conv_inputs(I.RESNET_STACK, li, s)
        say(f"stack layer {li + 1}: {s} fmt (5,{wi})->(5,{wa})->(5,{wo}) relu")
        d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, wi), (5, wa),
                         (5, wo), hf.ACT_RELU)
        pw = hf.pack(dev(w.reshape(-1, s.M)), (5, wi))
        out = hf.conv2d(planes, pw, d)
        got = conv_codes(hf, out, d, wo)
        qw = orc.quantize_f32(w, 5, wi)
        pts = sample_points((s.N, s.OH, s.OW), s.M, np.random.default_rng([3, li]), SAMPLES)
        want = orc.conv2d_points(in_codes, qw, pts, s.stride, s.pad, 5, wi, wa, wo, act=1)
        bad = np.flatnonzero(got[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]] != want)
        assert bad.size == 0, f"layer {li + 1}: {bad.size} mismatches; first at {pts[bad[0]]}"
        # sanity of the workload itself: ReLU outputs are never negative
        sign = (got >> np.uint64(5 + wo)) & np.uint64(1)
        assert not sign.any()
        planes, in_codes = out, got
