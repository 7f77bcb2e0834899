"""Seeded synthetic inputs for the HOBFLOPS workloads.

This module only draws random numbers: it holds none of the number format's
arithmetic, so the GPU path and the CPU oracle can both take their inputs from
it. Every tensor comes from ``numpy.random.default_rng([workload, tensor,
variant])`` (tensor 0 = IFM or a, 1 = weights or b, 2 = c, 3 = exception mask),
is drawn in float64 and cast to float32; that float32 tensor is what both sides
quantize. Layouts: IFM NHWC, weights HWIO (KH, KW, C, M).

The paper's own workload is a MobileNets-shaped layer (Sec. 3.4 and Sec. 4);
no dataset or trained weights are involved, so value distributions stand in
for real activations and weights.
"""
from dataclasses import dataclass

import numpy as np

# Workload ids used in the seeds.
SMALL_CONV, FMA_SWEEP, RESNET_CONV, MANTISSA_SWEEP, RESNET_STACK, TYPE_SWEEP = 0, 1, 2, 3, 4, 5

# Formats of the element-wise a*b+c sweep: (wE, wF) of the operands; the result
# has one more fraction bit (the paper's "single" MAC type, Table 3).
FMA_FORMATS = [(4, 2), (5, 3), (5, 5), (5, 7), (5, 10), (8, 7)]
MANTISSA_SWEEP_WF = list(range(2, 11))


@dataclass(frozen=True)
class ConvShape:
    N: int
    H: int
    W: int
    C: int
    M: int
    KH: int
    KW: int
    stride: int
    pad: int

    @property
    def OH(self):
        return (self.H + 2 * self.pad - self.KH) // self.stride + 1

    @property
    def OW(self):
        return (self.W + 2 * self.pad - self.KW) // self.stride + 1

    @property
    def macs(self):
        return self.N * self.OH * self.OW * self.M * self.KH * self.KW * self.C


SMALL_CONV_SHAPE = ConvShape(1, 8, 8, 4, 8, 3, 3, 1, 1)
RESNET_CONV_SHAPE = ConvShape(8, 56, 56, 64, 64, 3, 3, 1, 1)
MANTISSA_SWEEP_SHAPES = [ConvShape(4, 224, 224, 3, 64, 3, 3, 1, 1),
                         ConvShape(4, 28, 28, 256, 512, 3, 3, 1, 1)]


def mobilenet_layer(batch):
    """The layer the paper's type sweep runs on (Sec. 3.4 and Sec. 4): the
    "Conv dw / s2" position of MobileNets, 14x14x512 input, 3x3 kernels,
    stride 2. Taken here as a dense MCMK conv with M = 512 and pad 1 (the
    paper gives neither M nor the padding)."""
    return ConvShape(batch, 14, 14, 512, 512, 3, 3, 2, 1)


def resnet_stack_shapes(batch=16):
    """The 13-layer ResNet-shaped stack: (kernel, Cin, Cout, stride, pad) per layer."""
    spec = [(3, 64, 64, 1, 1), (3, 64, 64, 1, 1), (1, 64, 128, 2, 0),
            (3, 128, 128, 1, 1), (3, 128, 128, 1, 1), (3, 128, 256, 2, 1),
            (3, 256, 256, 1, 1), (1, 256, 256, 1, 0), (3, 256, 256, 1, 1),
            (3, 256, 512, 2, 1), (3, 512, 512, 1, 1), (1, 512, 512, 1, 0),
            (3, 512, 512, 1, 1)]
    shapes, h = [], 56
    for k, cin, cout, s, p in spec:
        sh = ConvShape(batch, h, h, cin, cout, k, k, s, p)
        shapes.append(sh)
        h = sh.OH
    return shapes


def resnet_stack_formats(nlayers=13):
    """(wF_in, wF_acc, wF_out) per layer, wE = 5: odd layers (1-based) take
    (5,3) inputs, even layers (5,5); each layer's output feeds the next layer's
    input format, and the last layer outputs its accumulator format."""
    wf_in = [3 if (i % 2 == 0) else 5 for i in range(nlayers)]
    out = []
    for i in range(nlayers):
        acc = wf_in[i] + 1
        nxt = wf_in[i + 1] if i + 1 < nlayers else acc
        out.append((wf_in[i], acc, nxt))
    return out


def rng(workload, tensor, variant=0, *extra):
    return np.random.default_rng([workload, tensor, variant, *extra])


def uniform(g, shape, lo, hi):
    return g.uniform(lo, hi, size=shape).astype(np.float32)


def relu_like(g, shape):
    """|N(0,1)| with each entry zeroed with probability 1/2."""
    v = np.abs(g.standard_normal(size=shape))
    v[g.random(size=shape) < 0.5] = 0.0
    return v.astype(np.float32)


def normal(g, shape, std):
    return (g.standard_normal(size=shape) * std).astype(np.float32)


def inject_specials(x, g, frac=0.01):
    """Replace a fraction of entries by +-0, +-inf or NaN (uniform kind, random sign)."""
    x = x.copy()
    sel = np.flatnonzero(g.random(size=x.size) < frac)
    kind = g.integers(0, 3, size=sel.size)
    sign = np.where(g.random(size=sel.size) < 0.5, -1.0, 1.0)
    vals = np.where(kind == 0, 0.0 * sign, np.where(kind == 1, np.inf * sign, np.nan))
    x.reshape(-1)[sel] = vals.astype(np.float32)
    return x


def small_conv_inputs():
    """8x8x4 IFM, eight 3x3x4 kernels, values U[-1,1]."""
    s = SMALL_CONV_SHAPE
    ifm = uniform(rng(SMALL_CONV, 0), (s.N, s.H, s.W, s.C), -1.0, 1.0)
    w = uniform(rng(SMALL_CONV, 1), (s.KH, s.KW, s.C, s.M), -1.0, 1.0)
    return ifm, w


def fma_operands(variant, n=1 << 24):
    """a, b, c for the element-wise sweep: U[-4,4] with 1% special values each."""
    out = []
    for t in range(3):
        v = uniform(rng(FMA_SWEEP, t, variant), (n,), -4.0, 4.0)
        out.append(inject_specials(v, rng(FMA_SWEEP, 3, variant, t)))
    return tuple(out)


def conv_inputs(workload, variant, shape: ConvShape, w_std=None):
    """ReLU-like IFM and N(0, w_std) weights; w_std defaults to sqrt(2/fan_in)."""
    s = shape
    if w_std is None:
        w_std = float(np.sqrt(2.0 / (s.KH * s.KW * s.C)))
    ifm = relu_like(rng(workload, 0, variant), (s.N, s.H, s.W, s.C))
    w = normal(rng(workload, 1, variant), (s.KH, s.KW, s.C, s.M), w_std)
    return ifm, w


def resnet_conv_inputs():
    return conv_inputs(RESNET_CONV, 0, RESNET_CONV_SHAPE, w_std=0.05)


def mantissa_sweep_inputs(shape_index, wF):
    """The mantissa sweep's layers take the ResNet layer's value distributions:
    ReLU-like IFM, weights N(0, 0.05)."""
    return conv_inputs(MANTISSA_SWEEP, 16 * shape_index + wF, MANTISSA_SWEEP_SHAPES[shape_index],
                       w_std=0.05)


def type_sweep_inputs(batch):
    """Inputs of the MobileNets-shaped layer of the type sweep: ReLU-like IFM,
    weights N(0, sqrt(2/fan_in)) (an initialised layer of 4,608 taps)."""
    return conv_inputs(TYPE_SWEEP, 0, mobilenet_layer(batch))


def random_codes(seed, shape, nbits):
    """Raw codes with every one of the low nbits drawn at random (this includes
    non-canonical special values) -- for exercising code inputs."""
    g = np.random.default_rng([99, seed])
    return g.integers(0, 1 << nbits, size=shape, dtype=np.uint64).astype(np.uint32)
