"""GPU parity at the workloads' full sizes, on sampled outputs.

Each workload runs whole on the GPU through the C ABI, at its real shape:
  * the element-wise a*b+c sweep: 2^24 triples per format, six formats;
  * the mantissa sweep: 4x224x224x3 -> 64 and 4x28x28x256 -> 512, 3x3, for
    input formats (5, m), m = 2..10, accumulating in (5, m+1);
  * the 13-layer ResNet-shaped stack at batch 16, planes kept on the GPU from
    layer to layer, ReLU and a format change in every epilogue.
The oracle then recomputes a seeded sample of the outputs one by one (every
border position of every image plus random points) and the codes must agree
bit for bit. For the stack the oracle's input to each layer is the GPU's own
output of the previous layer (teacher forcing), so every layer is checked on
its own; the first layer's input and all weights are quantised by the oracle.
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
def test_fma_sweep_full_size(idx):
    """2^24 triples, U[-4,4] with 1 % specials per operand: all computed on the
    GPU, 2^20 random ones plus the last 4,096 recomputed by the oracle."""
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
    g = np.random.default_rng([1, idx])
    sel = np.unique(np.concatenate([g.integers(0, n, 1 << 20), np.arange(n - 4096, n)]))
    qa, qb, qc = (threaded(orc.quantize_f32, t[sel], fixed=(wE, wF)) for t in (a, b, c))
    want = threaded(orc.muladd, qa, qb, qc, fixed=(wE, wF, wa))
    bad = np.flatnonzero(got[sel] != want)
    assert bad.size == 0, f"{bad.size} mismatches of {sel.size}; first at {sel[bad[0]]}"
    want_f = orc.decode_f32(want, wE, wa).view(np.uint32)
    assert np.array_equal(got_f[sel], want_f)


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
    ifm, w = I.conv_inputs(I.MANTISSA_SWEEP, 16 * si + m, s)
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
