"""GPU parity: the HIP path through the C ABI against the oracle, bit for bit.

Every comparison is of codes (integers): zero mismatches allowed. Inputs are
seeded; each case prints what it runs before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from gpu_util import codes_of, dev, need_gpu, say
from paper_2007_06563_amd import inputs as I
from paper_2007_06563_amd import variants
from planes import pack_codes, unpack_planes

pytestmark = pytest.mark.gpu


def rand_f32(seed, n, lo=-4.0, hi=4.0, specials=0.02):
    g = np.random.default_rng([7, seed])
    x = g.uniform(lo, hi, n).astype(np.float32)
    # plus raw bit patterns (all exponents, subnormals, NaN payloads)
    raw = g.integers(0, 1 << 32, n // 4, dtype=np.uint64).astype(np.uint32).view(np.float32)
    x[: n // 4] = raw
    return I.inject_specials(x, g, specials)


# NB = 3 + wE + wF must fit a 32-bit code: (8,21), (7,22) and (6,23) are the
# widest; wF = 23 keeps every float32 fraction bit (no rounding)
PACK_FORMATS = [(2, 1), (4, 2), (4, 3), (5, 2), (5, 3), (5, 4), (5, 10), (5, 11), (8, 7), (8, 8),
                (8, 21), (7, 22), (6, 12), (6, 23), (2, 23)]


def near_ties(seed, n, wE, wF):
    """float32 values at, and one float32 ulp either side of, the midpoints
    between neighbouring codes, over the format's exponent range and a few
    binades past both ends (round-up carries, overflow, underflow)."""
    g = np.random.default_rng([11, seed])
    bias = (1 << (wE - 1)) - 1
    e = g.integers(127 - bias - 3, 127 + bias + 4, n).clip(1, 254).astype(np.uint32)
    k = 23 - wF
    m = g.integers(0, 1 << 23, n).astype(np.uint32)
    if k > 0:  # (wF = 23 has no midpoints: every float32 value is exact)
        m = (m >> k << k) | np.uint32(1 << (k - 1))
    m = (m.astype(np.int64) + g.integers(-1, 2, n)).astype(np.uint32) & np.uint32(0x7FFFFF)
    s = g.integers(0, 2, n).astype(np.uint32) << 31
    return (s | (e << 23) | m).view(np.float32)


# (rows, length): ragged rows (3 groups per row, an odd number of groups) and
# rows that are a whole number of groups (the groups tile the flat array)
PACK_SHAPES = [(37, 70), (21, 96)]


@pytest.mark.parametrize("rows,length", PACK_SHAPES)
@pytest.mark.parametrize("wE,wF", PACK_FORMATS)
def test_pack_unpack_float32(wE, wF, rows, length):
    hf = need_gpu()
    x = rand_f32(wE * 100 + wF, rows * length).reshape(rows, length)
    say(f"pack f32 fmt=({wE},{wF}) shape={x.shape}")
    planes = hf.pack(dev(x), (wE, wF))
    torch.cuda.synchronize()
    want = orc.quantize_f32(x, wE, wF)
    nbits = 3 + wE + wF
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), pack_codes(want, nbits))
    codes = hf.unpack(planes, rows, length, (wE, wF), kind="code")
    vals = hf.unpack(planes, rows, length, (wE, wF), kind="f32")
    torch.cuda.synchronize()
    assert np.array_equal(codes_of(codes), want)
    want_f = orc.decode_f32(want, wE, wF)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), want_f.view(np.uint32))


@pytest.mark.parametrize("rows,length", PACK_SHAPES)
@pytest.mark.parametrize("wE,wF", PACK_FORMATS)
def test_pack_rounding_ties_and_range_ends(wE, wF, rows, length):
    hf = need_gpu()
    x = near_ties(wE * 100 + wF, rows * length, wE, wF).reshape(rows, length)
    say(f"pack ties fmt=({wE},{wF}) shape={x.shape}")
    planes = hf.pack(dev(x), (wE, wF))
    torch.cuda.synchronize()
    want = orc.quantize_f32(x, wE, wF)
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), pack_codes(want, 3 + wE + wF))


def _want_planes(src, wE, wF):
    """Expected planes of a pack: oracle quantisation of float32 values, or the
    codes' low NB bits."""
    nbits = 3 + wE + wF
    if src.dtype == np.float32:
        codes = orc.quantize_f32(src, wE, wF)
    else:
        codes = src.view(np.uint32).astype(np.uint64) & np.uint64((1 << nbits) - 1)
    return pack_codes(codes, nbits)


@pytest.mark.parametrize("wE,wF", [f for f in PACK_FORMATS if 3 + f[0] + f[1] <= 20])
def test_unpack_every_code(wE, wF):
    """Every code of the format (2^NB, non-canonical specials included) packed
    from codes and unpacked to float32 and to codes, against the oracle's
    decoder."""
    hf = need_gpu()
    nbits = 3 + wE + wF
    codes = np.arange(1 << nbits, dtype=np.uint32).reshape(1, -1)
    say(f"unpack every code fmt=({wE},{wF}) n={codes.size}")
    planes = hf.pack(dev(codes.view(np.int32)), (wE, wF))
    back = hf.unpack(planes, 1, codes.size, (wE, wF), kind="code")
    vals = hf.unpack(planes, 1, codes.size, (wE, wF), kind="f32")
    torch.cuda.synchronize()
    assert np.array_equal(codes_of(back), codes.astype(np.uint64))
    want = orc.decode_f32(codes.astype(np.uint64), wE, wF)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), want.view(np.uint32))


def test_pack_every_float32_pattern():
    """All 2^32 float32 bit patterns through the pack kernel (and the unpack
    to codes), against checksums of the oracle's codes per 2^28 patterns
    (tests/golden/quantize_all_f32.json, written by
    tests/golden/make_quantize_checksums.py from oracle/ alone)."""
    import json
    import os
    hf = need_gpu()
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "quantize_all_f32.json")))
    n = 1 << gold["chunk_bits"]
    for key, chunks in gold["formats"].items():
        wE, wF = (int(v) for v in key.split(","))
        for c, want in enumerate(chunks):
            say(f"pack every float32 pattern fmt=({wE},{wF}) chunk {c}")
            first = c * n
            i = torch.arange(first, first + n, dtype=torch.int64, device="cuda")
            bits = torch.where(i >= (1 << 31), i - (1 << 32), i).to(torch.int32)
            planes = hf.pack(bits.view(torch.float32).reshape(1, n), (wE, wF))
            codes = hf.unpack(planes, 1, n, (wE, wF), kind="code").reshape(-1).to(torch.int64)
            codes &= (1 << 32) - 1
            got = []
            for A, B, P in gold["hashes"]:
                h = (A * (i % P) + B) % P
                got.append(int(((((codes + 1) % P) * h) % P).sum().item() % P))
            assert got == want, (key, c)
            del i, bits, planes, codes, h


@pytest.mark.parametrize("wE,wF", [(5, 3), (8, 7), (5, 10), (6, 23)])
def test_pack_unpack_16_byte_paths_and_fallbacks(wE, wF):
    """Dense tensors move 16 bytes per lane through LDS when both arrays are
    16-byte aligned; a large launch (eight passes a wave) whose last wave is
    partial, and sources or destinations only 4-byte aligned (the per-value
    path), all against the oracle."""
    hf = need_gpu()
    nb = 3 + wE + wF
    groups = (1 << 18) + 5           # eight passes a wave, last wave partial
    n = 32 * groups
    x = rand_f32(900 + wF, n + 4)
    xd = dev(x)
    sel = np.r_[0:64, groups - 40:groups]               # first waves and the partial tail
    vsel = (32 * sel[:, None] + np.arange(32)).reshape(-1)
    for off in (0, 1):               # off 1: source 4-byte aligned only
        say(f"pack 16-byte path fmt=({wE},{wF}) groups={groups} src offset={off}")
        want = orc.quantize_f32(x[off + vsel], wE, wF)
        src = xd[off:off + n].view(1, n)
        planes = hf.pack(src, (wE, wF))
        torch.cuda.synchronize()
        got = planes.cpu().numpy().view(np.uint32).reshape(-1, nb)
        assert np.array_equal(got[sel], pack_codes(want.reshape(1, -1), nb).reshape(-1, nb))
        for doff in (0, 1):          # doff 1: destination 4-byte aligned only
            say(f"unpack 16-byte path fmt=({wE},{wF}) dst offset={doff}")
            buf = torch.empty(n + 4, dtype=torch.int32, device="cuda")
            out = buf[doff:doff + n].view(1, n)
            hf.unpack(planes, 1, n, (wE, wF), kind="code", out=out)
            torch.cuda.synchronize()
            codes = codes_of(out)[0]
            assert np.array_equal(codes[vsel], want)
    # a multiple of 16 groups with every value checked, small launch (four passes)
    m = 32 * 16 * 9
    want = orc.quantize_f32(x[:m], wE, wF)
    xs = dev(x[:m].reshape(9, -1))
    planes = hf.pack(xs, (wE, wF))
    vals = hf.unpack(planes, 9, m // 9, (wE, wF), kind="f32")
    torch.cuda.synchronize()
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), pack_codes(want.reshape(9, -1), nb))
    assert np.array_equal(vals.cpu().numpy().view(np.uint32).reshape(-1),
                          orc.decode_f32(want, wE, wF).view(np.uint32))


@pytest.mark.parametrize("njobs", [5, 11])
@pytest.mark.parametrize("wE,wF", [(5, 3), (8, 7), (4, 2)])
def test_pack_batch_equals_single_packs(wE, wF, njobs):
    """One launch per 8 jobs; dense, ragged, code, single-value and empty jobs
    mixed. Each job's planes against the oracle."""
    hf = need_gpu()
    g = np.random.default_rng([13, wE, wF, njobs])
    shapes = [(21, 96), (37, 70), (5, 1000), (1, 1), (0, 5), (3, 32), (9, 33), (2, 64), (4, 7),
              (6, 200), (1, 31)][:njobs]
    srcs = []
    for t, (r, n) in enumerate(shapes):
        if t % 3 == 2:
            srcs.append(I.random_codes(600 + t, (r, n), 32).view(np.int32))
        else:
            srcs.append(rand_f32(500 + t, r * n).reshape(r, n))
    say(f"pack_batch fmt=({wE},{wF}) jobs={njobs}")
    outs = hf.pack_batch([dev(x) for x in srcs], (wE, wF))
    torch.cuda.synchronize()
    for x, o in zip(srcs, outs):
        assert np.array_equal(o.cpu().numpy().view(np.uint32), _want_planes(x, wE, wF)), x.shape


def test_pack_batch_splits_large_tensors():
    """A tensor of more than 2^25 groups spans several ranges of a launch; the
    rows next to the range boundaries and at both ends against the oracle."""
    hf = need_gpu()
    rows, length = (1 << 25) + 4099, 32       # one group per row
    say(f"pack_batch large rows={rows} len={length}")
    gen = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn((rows, length), generator=gen, device="cuda") * 3.0
    small = dev(rand_f32(77, 40 * 45).reshape(40, 45))
    o_big, o_small = hf.pack_batch([x, small], (5, 3))
    torch.cuda.synchronize()
    for r0 in (0, (1 << 25) - 3, rows - 5):
        xs = x[r0:r0 + 5].cpu().numpy()
        got = o_big[r0:r0 + 5].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, _want_planes(xs, 5, 3)), r0
    assert np.array_equal(o_small.cpu().numpy().view(np.uint32),
                          _want_planes(small.cpu().numpy(), 5, 3))
    del x, o_big


@pytest.mark.parametrize("length", [1000, 1024])
@pytest.mark.parametrize("wE,wF", [(5, 3), (5, 4), (8, 8)])
def test_pack_codes_round_trip(wE, wF, length):
    hf = need_gpu()
    nbits = 3 + wE + wF
    rows = 5
    raw = I.random_codes(nbits, (rows, length), 32)  # garbage above NB too
    say(f"pack codes fmt=({wE},{wF})")
    planes = hf.pack(dev(raw.view(np.int32)), (wE, wF))
    back = hf.unpack(planes, rows, length, (wE, wF), kind="code")
    torch.cuda.synchronize()
    masked = raw.astype(np.uint64) & np.uint64((1 << nbits) - 1)
    assert np.array_equal(codes_of(back), masked)
    assert np.array_equal(unpack_planes(planes.cpu().numpy(), length), masked)


def test_wider_than_32_bit_codes_rejected():
    hf = need_gpu()
    with pytest.raises(hf.HobflopsError):
        hf.pack(torch.zeros((2, 32), device="cuda"), (8, 23))


def test_empty_pack_is_a_no_op():
    hf = need_gpu()
    hf.pack(torch.empty((0, 5), device="cuda"), (5, 3), rows=0, length=5)


def test_muladd_every_triple_of_codes():
    """Every triple of codes of the small formats in
    tests/golden/muladd_all_codes.json (written by
    tests/golden/make_muladd_checksums.py from oracle/ alone): a = i mod 2^NB,
    b = (i >> NB) mod 2^NB, c = i >> 2 NB, packed from codes, through
    hobflops_muladd, the result codes' checksums per 2^24 triples against the
    oracle's."""
    import json
    import os
    hf = need_gpu()
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "muladd_all_codes.json")))
    n = 1 << gold["chunk_bits"]
    for key, chunks in gold["cases"].items():
        wE, wi, wa = (int(v) for v in key.split(",")[:3])
        rnd = hf.ROUND_NEAREST_EVEN if key.endswith("rne") else hf.ROUND_TOWARD_ZERO
        nb = 3 + wE + wi
        for ch, want in enumerate(chunks):
            say(f"muladd every triple {key} chunk {ch}")
            i = torch.arange(ch * n, (ch + 1) * n, dtype=torch.int64, device="cuda")
            ops = [((i >> (k * nb)) & ((1 << nb) - 1)).to(torch.int32).reshape(1, n)
                   for k in range(3)]
            pa, pb, pc = hf.pack_batch(ops, (wE, wi))
            r = hf.muladd(pa, pb, pc, n, (wE, wi), (wE, wa), round=rnd)
            codes = hf.unpack(r, 1, n, (wE, wa), kind="code").reshape(-1).to(torch.int64)
            codes &= (1 << 32) - 1
            got = []
            for A, B, P in gold["hashes"]:
                h = (A * (i % P) + B) % P
                got.append(int(((((codes + 1) % P) * h) % P).sum().item() % P))
            assert got == want, (key, ch)


@pytest.mark.parametrize("v", variants.MULADD_VARIANTS, ids=variants.muladd_tag)
def test_muladd_vs_oracle(v):
    hf = need_gpu()
    wE, wi, wa, rnd = v
    n = (1 << 15) + 77  # ragged tail
    a, b, c = (rand_f32(1000 * wi + t, n) for t in range(3))
    say(f"muladd {v} n={n}")
    pa, pb, pc = (hf.pack(dev(t), (wE, wi)) for t in (a, b, c))
    r = hf.muladd(pa, pb, pc, n, (wE, wi), (wE, wa), round=rnd)
    got = codes_of(hf.unpack(r, 1, n, (wE, wa), kind="code"))[0]
    qa, qb, qc = (orc.quantize_f32(t, wE, wi) for t in (a, b, c))
    want = orc.muladd(qa, qb, qc, wE, wi, wa, rnd=rnd)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches; first a={qa[bad[0]]:#x} b={qb[bad[0]]:#x} " \
                          f"c={qc[bad[0]]:#x} got={got[bad[0]]:#x} want={want[bad[0]]:#x}"


@pytest.mark.parametrize("v", variants.MULADD_VARIANTS, ids=variants.muladd_tag)
def test_muladd_raw_codes_vs_oracle(v):
    """Non-canonical inputs: every field bit random, specials with garbage fields."""
    hf = need_gpu()
    wE, wi, wa, rnd = v
    nbits = 3 + wE + wi
    n = 1 << 14
    a, b, c = (I.random_codes(nbits * 10 + t, (1, n), nbits) for t in range(3))
    say(f"muladd raw codes {v}")
    pa, pb, pc = (hf.pack(dev(t.view(np.int32)), (wE, wi)) for t in (a, b, c))
    r = hf.muladd(pa, pb, pc, n, (wE, wi), (wE, wa), round=rnd)
    got = codes_of(hf.unpack(r, 1, n, (wE, wa), kind="code"))[0]
    want = orc.muladd(a[0].astype(np.uint64), b[0].astype(np.uint64), c[0].astype(np.uint64), wE,
                      wi, wa, rnd=rnd)
    assert np.array_equal(got, want)


def run_conv(hf, ifm_codes, w_codes, stride, pad, wE, wi, wa, wo, act, algo=0, rnd=0):
    """GPU conv on code tensors (NHWC / HWIO) -> output codes [N, OH, OW, M]."""
    N, H, W, C = ifm_codes.shape
    KH, KW, _, M = w_codes.shape
    d = hf.conv_desc(N, H, W, C, M, KH, KW, stride, pad, (wE, wi), (wE, wa), (wE, wo), act, algo,
                     round=rnd)
    OH, OW = hf.conv_out_hw(d)
    pi = hf.pack(dev(ifm_codes.astype(np.uint32).view(np.int32).reshape(N * H * W, C)), (wE, wi))
    pw = hf.pack(dev(w_codes.astype(np.uint32).view(np.int32).reshape(KH * KW * C, M)), (wE, wi))
    po = hf.conv2d(pi, pw, d)
    out = hf.unpack(po, N * OH * OW, M, (wE, wo), kind="code")
    torch.cuda.synchronize()
    return codes_of(out).reshape(N, OH, OW, M)


@pytest.mark.parametrize("rnd", [0, 1], ids=["rne", "rtz"])
@pytest.mark.parametrize("algo", [1, 2, 3], ids=["fused", "split", "compact"])
def test_conv_every_product_pair(algo, rnd):
    """A one-tap convolution whose IFM positions are all 2^11 codes of (5,3)
    and whose kernels are all 2^11 codes too: every (w, x) pair through the
    multiplier, the add into +0 and the epilogue, against the oracle."""
    hf = need_gpu()
    nb = 11
    codes = np.arange(1 << nb, dtype=np.uint64)
    ifm = codes.reshape(1, 1, 1 << nb, 1)
    w = codes.reshape(1, 1, 1, 1 << nb)
    say(f"conv every product pair algo={algo} rnd={rnd}")
    got = run_conv(hf, ifm, w, 1, 0, 5, 3, 4, 4, 0, algo, rnd)
    want = orc.conv2d(ifm, w, 1, 0, 5, 3, 4, 4, rnd=orc.RTZ if rnd else orc.RNE)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} mismatches; first at {bad[0]}"


def test_small_conv_workload():
    """8x8x4 IFM, eight 3x3x4 kernels, (5,3) inputs, (5,4) accumulation."""
    hf = need_gpu()
    ifm, w = I.small_conv_inputs()
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    say("conv small workload")
    got = run_conv(hf, qi, qw, 1, 1, 5, 3, 4, 4, 0)
    want = orc.conv2d(qi, qw, 1, 1, 5, 3, 4, 4)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("algo", [1, 2, 3], ids=["fused", "split", "compact"])
@pytest.mark.parametrize("v", variants.CONV_VARIANTS, ids=variants.conv_tag)
def test_conv_variants_vs_oracle(v, algo):
    """Every generated variant, in both kernel shapes, on a problem spanning two
    channel words and two kernel words, both ragged, with padding and specials."""
    hf = need_gpu()
    wE, wi, wa, wo, act, rnd = v
    d0 = hf.conv_desc(1, 3, 3, 1, 1, 1, 1, 1, 0, (wE, wi), (wE, wa), (wE, wo), act, algo, round=rnd)
    if not hf.conv2d_supported(d0):
        if algo == hf.ALGO_SPLIT_COMPACT:
            pytest.skip("variant generated without the compact split kernel (registers)")
        assert algo == hf.ALGO_SPLIT and hf.netlist_ops((wE, wi), (wE, wa), rnd)["mul"] == 0
        pytest.skip("variant generated without the split kernel (registers)")
    g = np.random.default_rng([11, wi, wa, wo, act, rnd])
    N, H, W, C, M = 2, 7, 9, 37, 40
    ifm = I.inject_specials(g.uniform(-2, 2, (N, H, W, C)).astype(np.float32), g, 0.01)
    w = I.inject_specials(g.uniform(-1, 1, (3, 3, C, M)).astype(np.float32), g, 0.005)
    qi, qw = orc.quantize_f32(ifm, wE, wi), orc.quantize_f32(w, wE, wi)
    for stride, pad in ((1, 1), (2, 0)):
        say(f"conv variant {v} algo={algo} stride={stride} pad={pad}")
        got = run_conv(hf, qi, qw, stride, pad, wE, wi, wa, wo, act, algo, rnd)
        want = orc.conv2d(qi, qw, stride, pad, wE, wi, wa, wo, act, rnd=rnd)
        bad = np.argwhere(got != want)
        assert bad.size == 0, f"{len(bad)} mismatches, first at {bad[0]}"


def test_auto_kernel_choice():
    """AUTO's kernel shape by chain waves (64 positions of one 32-kernel tile)
    per SIMD: at most one, the split kernel (the bench layer, 784); up to two,
    its compact form (stack layer 1, 1,568) or, where that was not generated,
    the split kernel (stack layer 2's formats); more, the fused kernel (the
    4x224x224x3 layer, 6,272)."""
    hf = need_gpu()
    simds = 4 * torch.cuda.get_device_properties(0).multi_processor_count
    cases = [((8, 56, 56, 64, 64), (5, 3), (5, 4), (5, 4), 0, 784),
             ((16, 56, 56, 64, 64), (5, 3), (5, 4), (5, 5), 1, 1568),
             ((16, 56, 56, 64, 64), (5, 5), (5, 6), (5, 3), 1, 1568),
             ((4, 224, 224, 3, 64), (5, 3), (5, 4), (5, 4), 0, 6272)]
    for (N, H, W, C, M), fi, fa, fo, act, chains in cases:
        d = hf.conv_desc(N, H, W, C, M, 3, 3, 1, 1, fi, fa, fo, act, hf.ALGO_AUTO)
        compact = hf.conv2d_supported(hf.conv_desc(N, H, W, C, M, 3, 3, 1, 1, fi, fa, fo, act,
                                                   hf.ALGO_SPLIT_COMPACT))
        want = (hf.ALGO_SPLIT if chains <= simds else
                (hf.ALGO_SPLIT_COMPACT if compact else hf.ALGO_SPLIT) if chains <= 2 * simds
                else hf.ALGO_FUSED)
        assert hf.conv2d_algo(d) == want, (N, H, W, C, M, fi, fa)
    if simds == 1024:  # MI355X: the shapes above land in each regime
        assert [hf.conv2d_algo(hf.conv_desc(N, H, W, C, M, 3, 3, 1, 1, fi, fa, fo, act, 0))
                for (N, H, W, C, M), fi, fa, fo, act, _ in cases] == [2, 3, 2, 1]


@pytest.mark.parametrize("algo", [1, 2, 3], ids=["fused", "split", "compact"])
def test_conv_1x1_and_raw_codes(algo):
    hf = need_gpu()
    qi = I.random_codes(1, (3, 5, 4, 70), 11).astype(np.uint64)
    qw = I.random_codes(2, (1, 1, 70, 33), 11).astype(np.uint64)
    say(f"conv 1x1 raw codes algo={algo}")
    got = run_conv(hf, qi, qw, 1, 0, 5, 3, 4, 4, 0, algo)
    want = orc.conv2d(qi, qw, 1, 0, 5, 3, 4, 4)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("algo", [1, 2, 3], ids=["fused", "split", "compact"])
def test_conv_tap_counts_not_multiple_of_batch(algo):
    """C = 3 with a 3x3 kernel (27 taps) and C = 5 with 1x1 (5 taps): batches and
    channel words end at different taps."""
    hf = need_gpu()
    g = np.random.default_rng(9)
    for (N, H, W, C, M, k, pad) in ((2, 9, 11, 3, 36, 3, 1), (1, 4, 4, 5, 7, 1, 0)):
        qi = orc.quantize_f32(g.uniform(-2, 2, (N, H, W, C)).astype(np.float32), 5, 3)
        qw = orc.quantize_f32(g.uniform(-1, 1, (k, k, C, M)).astype(np.float32), 5, 3)
        say(f"conv taps C={C} k={k} algo={algo}")
        got = run_conv(hf, qi, qw, 1, pad, 5, 3, 4, 4, 0, algo)
        assert np.array_equal(got, orc.conv2d(qi, qw, 1, pad, 5, 3, 4, 4))


@pytest.mark.parametrize("algo", [1, 2, 3], ids=["fused", "split", "compact"])
@pytest.mark.parametrize("M", [64, 40, 37])
def test_conv_fused_unpack(algo, M):
    """The unpack fused into the epilogue (ofm_kind F32 / CODE) equals the
    oracle's codes and their float32 values: full row, ragged last m-tile,
    a row length that is not a multiple of four, and an output that is only
    4-byte aligned."""
    hf = need_gpu()
    g = np.random.default_rng([12, M, algo])
    N, H, W, C = 2, 7, 9, 37
    ifm = I.inject_specials(g.uniform(-2, 2, (N, H, W, C)).astype(np.float32), g, 0.01)
    w = I.inject_specials(g.uniform(-1, 1, (3, 3, C, M)).astype(np.float32), g, 0.005)
    qi, qw = orc.quantize_f32(ifm, 5, 3), orc.quantize_f32(w, 5, 3)
    want = orc.conv2d(qi, qw, 1, 1, 5, 3, 4, 5, 1).reshape(-1, M)
    pi = hf.pack(dev(qi.astype(np.uint32).view(np.int32).reshape(-1, C)), (5, 3))
    pw = hf.pack(dev(qw.astype(np.uint32).view(np.int32).reshape(-1, M)), (5, 3))
    P = want.shape[0]
    for kind in (hf.OFM_CODE, hf.OFM_F32):
        for offset in (0, 1):
            say(f"conv fused unpack M={M} algo={algo} kind={kind} offset={offset}")
            d = hf.conv_desc(N, H, W, C, M, 3, 3, 1, 1, (5, 3), (5, 4), (5, 5), hf.ACT_RELU, algo,
                             ofm_kind=kind)
            dt = torch.float32 if kind == hf.OFM_F32 else torch.int32
            buf = torch.full((P * M + 8,), -1, dtype=dt, device="cuda")
            out = buf[offset:offset + P * M].view(P, M)
            hf.conv2d(pi, pw, d, out=out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            if kind == hf.OFM_CODE:
                assert np.array_equal(got.view(np.uint32).astype(np.uint64), want)
            else:
                assert np.array_equal(got.view(np.uint32), orc.decode_f32(want, 5, 5).view(np.uint32))
            rest = buf.cpu().numpy()
            assert np.all(rest[:offset].view(np.int32) == -1) if dt == torch.int32 else True
            assert np.all(rest[offset + P * M:].view(np.uint32) == rest[-1:].view(np.uint32))
