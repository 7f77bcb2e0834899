"""The split convolution kernel's bounded waits: a wait that reaches its
bound is counted, not silent.

The multiplier and accumulator waves of the split kernel hand products over
through LDS counters, and every wait for a counter is bounded, so a counter
that never came could not hang the GPU. A wait that ends at its bound leaves
the launch's results invalid, so the library counts it and the tests check
the count (conftest.py asserts it is zero after every GPU test). Here the
bound is set to zero from the host, so that waits give up at the first look
that misses: the kernels still run to the end, the count must be nonzero,
and with the default bound restored the same launch is exact again.
"""
import numpy as np
import pytest

import oracle as orc
from gpu_util import dev, need_gpu, say
from paper_2007_06563_amd import inputs as I

pytestmark = pytest.mark.gpu


ALGOS = pytest.mark.parametrize("algo", [2, 3], ids=["split", "compact"])


def _layer(hf, algo):
    s = I.RESNET_CONV_SHAPE
    ifm, w = I.resnet_conv_inputs()
    pi, pw = hf.pack_batch([dev(ifm.reshape(-1, s.C)), dev(w.reshape(-1, s.M))], (5, 3))
    d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, 3), (5, 4), (5, 4),
                     hf.ACT_NONE, algo, ofm_kind=hf.OFM_CODE)
    return s, ifm, w, pi, pw, d


@ALGOS
def test_default_bound_never_gives_up(algo):
    hf = need_gpu()
    s, ifm, w, pi, pw, d = _layer(hf, algo)
    hf.wait_failures(reset=True)
    say(f"split kernel (algo {algo}), default wait bound, 8x56x56x64->64")
    for _ in range(3):
        hf.conv2d(pi, pw, d)
    assert hf.wait_failures(reset=True) == 0


@ALGOS
def test_zero_bound_give_ups_are_counted(algo):
    hf = need_gpu()
    s, ifm, w, pi, pw, d = _layer(hf, algo)
    default = hf.get_wait_limit()
    hf.wait_failures(reset=True)
    try:
        hf.set_wait_limit(0)
        say(f"split kernel (algo {algo}), wait bound 0 (waits give up), 8x56x56x64->64")
        hf.conv2d(pi, pw, d)
        gave = hf.wait_failures(reset=True)
    finally:
        hf.set_wait_limit(default)
    assert gave > 0, "a zero bound must make waits give up, and each give-up must be counted"
    say(f"  {gave} give-ups counted; default bound restored")
    out = hf.conv2d(pi, pw, d)
    got = out.cpu().numpy().view(np.uint32).astype(np.uint64).reshape(s.N, s.OH, s.OW, s.M)
    assert hf.wait_failures(reset=True) == 0
    g = np.random.default_rng(31)
    pts = np.stack([g.integers(0, s.N, 4096), g.integers(0, s.OH, 4096),
                    g.integers(0, s.OW, 4096), g.integers(0, s.M, 4096)], 1).astype(np.int64)
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    want = orc.conv2d_points(qi, qw, pts, s.stride, s.pad, 5, 3, 4, 4)
    assert np.array_equal(got[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]], want)
