"""The generated netlists against the oracle, on the CPU.

The generator (gen/) builds each operator as a circuit, optimises and maps it
to 3-input LUTs, and allocates registers for the split kernel's assembly.
These tests evaluate the optimised circuits bit-parallel (gen/sim.py) on codes
-- random ones, with specials and non-canonical fields, and every code pair
where that is small -- and compare with the oracle's scalar results. The
register-allocated instruction lists are run by the allocator's interpreter
against the circuit itself. No GPU is involved.

The convolution's intermediate circuits (product, accumulating adder, fused
step) are non-canonical by design: a non-normal result is compared by its
exception field and sign only (and NaN by its exception field), which is how
every consumer reads it.
"""
import numpy as np
import pytest

import oracle
from paper_2007_06563_amd import build, variants
from paper_2007_06563_amd.gen import asmgen, fp, opt, regalloc, sim
from paper_2007_06563_amd.gen.regalloc import Block


def nbits(wE, wF):
    return 3 + wE + wF


def canon(codes, wE, wF):
    """Canonical form of codes (layout only): E = F = 0 unless normal, sign 0 for NaN."""
    c = np.asarray(codes, np.uint64)
    x = (c >> np.uint64(wE + wF + 1)) & np.uint64(3)
    s = (c >> np.uint64(wE + wF)) & np.uint64(1)
    ef = c & np.uint64((1 << (wE + wF)) - 1)
    ef = np.where(x == 1, ef, np.uint64(0))
    s = np.where(x == 3, np.uint64(0), s)
    return (x << np.uint64(wE + wF + 1)) | (s << np.uint64(wE + wF)) | ef


def random_codes(g, n, wE, wF):
    """Codes with every field random (non-canonical specials included), a
    quarter of them forced to a special exception value."""
    nb = nbits(wE, wF)
    c = g.integers(0, 1 << nb, size=n, dtype=np.uint64)
    special = g.random(n) < 0.25
    exn = g.integers(0, 4, size=n, dtype=np.uint64)
    top = np.uint64(wE + wF + 1)
    c = np.where(special, (c & np.uint64((1 << (wE + wF + 1)) - 1)) | (exn << top), c)
    return c


_OPT = {}
_SHIPPED = {"product_circuit": "prod", "accumulate_circuit": "accum", "mac_circuit": "mac"}


def optimized(kind, *args, **kw):
    """The optimised circuit of a builder, once per session: for the product,
    the accumulating adder and the fused step, exactly the library's
    (build.circuit, with its don't-care and resubstitution passes and the
    fused step composed from the other two; taken from the build's circuit
    cache when its sources match); otherwise opt.optimize of the builder's
    output."""
    key = (kind, args, tuple(sorted(kw.items())))
    if not _OPT:
        build._load_circuit_cache()  # the shipped circuits, where a build left them
    if key not in _OPT:
        if kind in _SHIPPED:
            _OPT[key] = build.circuit(_SHIPPED[kind], args, kw.get("rnd", "rne"))[0]
        else:
            _OPT[key] = opt.optimize(getattr(fp, kind)(*args, **kw))
    return _OPT[key]


def run(C, **ins):
    planes = {}
    for grp, lits in C.inputs:
        planes[grp] = sim.codes_to_planes(ins[grp], len(lits))
    out = sim.simulate(C, planes)
    return {grp: sim.planes_to_codes(v) for grp, v in out.items()}


N = 1 << 14


@pytest.mark.parametrize("v", variants.CONV_VARIANTS, ids=variants.conv_tag)
def test_conv_step_circuits(v):
    """Product, accumulating adder and fused step of every conv variant."""
    wE, wi, wa, wo, act, rnd = v
    r = variants.RND_NAME[rnd]
    g = np.random.default_rng([7, wE, wi, wa, rnd])
    w, x = random_codes(g, N, wE, wi), random_codes(g, N, wE, wi)
    acc = random_codes(g, N, wE, wa)
    p_ref = oracle.mul(w, x, wE, wi, wa, rnd=rnd)
    a_ref = oracle.add(acc, p_ref, wE, wa, rnd=rnd)
    p = run(optimized("product_circuit", wE, wi, wa, rnd=r), w=w, x=x)["p"]
    assert np.array_equal(canon(p, wE, wa), canon(p_ref, wE, wa))
    # the adder reads the product exactly as the multiplier leaves it
    a = run(optimized("accumulate_circuit", wE, wa, rnd=r), acc=acc, p=p)["acc"]
    assert np.array_equal(canon(a, wE, wa), canon(a_ref, wE, wa))
    m = run(optimized("mac_circuit", wE, wi, wa, rnd=r), acc=acc, w=w, x=x)["acc"]
    assert np.array_equal(canon(m, wE, wa), canon(a_ref, wE, wa))


@pytest.mark.parametrize("v", variants.CONV_VARIANTS, ids=variants.conv_tag)
def test_epilogue_circuits(v):
    """ReLU + convert of the accumulator into the output format: canonical."""
    wE, wi, wa, wo, act, rnd = v
    g = np.random.default_rng([8, wE, wa, wo, act, rnd])
    acc = random_codes(g, N, wE, wa)
    want = oracle.relu(acc, wE, wa) if act else acc
    want = oracle.convert(want, wE, wa, wo, rnd=rnd)
    C = optimized("convert_circuit", wE, wa, wo, relu=bool(act), rnd=variants.RND_NAME[rnd])
    got = run(C, a=acc)["r"]
    assert np.array_equal(got, want)


@pytest.mark.parametrize("v", variants.MULADD_VARIANTS, ids=variants.muladd_tag)
def test_muladd_circuits(v):
    wE, wi, wa, rnd = v
    g = np.random.default_rng([9, wE, wi, wa, rnd])
    a, b, c = (random_codes(g, N, wE, wi) for _ in range(3))
    want = oracle.muladd(a, b, c, wE, wi, wa, rnd=rnd)
    got = run(optimized("muladd_circuit", wE, wi, wa, rnd=variants.RND_NAME[rnd]), a=a, b=b, c=c)["r"]
    assert np.array_equal(got, want)


@pytest.mark.parametrize("rnd", [variants.RNE, variants.RTZ], ids=["rne", "rtz"])
def test_small_adder_every_pair(rnd):
    """Every pair of (4,2) codes (512 x 512) through the optimised adder."""
    wE, wF = 4, 2
    nb = nbits(wE, wF)
    allc = np.arange(1 << nb, dtype=np.uint64)
    a = np.repeat(allc, 1 << nb)
    b = np.tile(allc, 1 << nb)
    want = oracle.add(a, b, wE, wF, rnd=rnd)
    got = run(optimized("accumulate_circuit", wE, wF, rnd=variants.RND_NAME[rnd]), acc=a, p=b)["acc"]
    assert np.array_equal(canon(got, wE, wF), canon(want, wE, wF))


@pytest.mark.parametrize("rnd", [variants.RNE, variants.RTZ], ids=["rne", "rtz"])
@pytest.mark.parametrize("wFo", [3, 5])
def test_small_multiplier_every_pair(rnd, wFo):
    wE, wF = 4, 2
    nb = nbits(wE, wF)
    allc = np.arange(1 << nb, dtype=np.uint64)
    a = np.repeat(allc, 1 << nb)
    b = np.tile(allc, 1 << nb)
    want = oracle.mul(a, b, wE, wF, wFo, rnd=rnd)
    got = run(optimized("product_circuit", wE, wF, wFo, rnd=variants.RND_NAME[rnd]), w=a, x=b)["p"]
    assert np.array_equal(canon(got, wE, wFo), canon(want, wE, wFo))


def test_resynthesis_keeps_function():
    """Window resynthesis changes structure, never the function."""
    C = opt.sweep(fp.accumulate_circuit(5, 4))
    D = opt.resynthesize(opt.lut_map(opt.functional_reduce(C)))
    g = np.random.default_rng(3)
    acc, p = random_codes(g, N, 5, 4), random_codes(g, N, 5, 4)
    assert np.array_equal(run(C, acc=acc, p=p)["acc"], run(D, acc=acc, p=p)["acc"])


def test_resubstitution_keeps_cared_outputs():
    """Resubstitution under the non-canonical don't-cares removes LUTs of the
    (2,2) adder and changes no output bit that a consumer reads, on every
    pair of codes."""
    wE, wF = 2, 2
    care = opt.noncanonical_care(wE, wF)
    C = opt.optimize(fp.accumulate_circuit(wE, wF))
    D = opt.resubstitute(C, care)
    assert D.n_nodes() < C.n_nodes()
    nb = nbits(wE, wF)
    allc = np.arange(1 << nb, dtype=np.uint64)
    a, b = np.repeat(allc, 1 << nb), np.tile(allc, 1 << nb)
    got, want = run(D, acc=a, p=b)["acc"], run(C, acc=a, p=b)["acc"]
    assert np.array_equal(canon(got, wE, wF), canon(want, wE, wF))


def test_decompose2_examples():
    """g(h(S), T) decompositions of hand-made 4- and 5-input functions."""
    from paper_2007_06563_amd.gen.circuit import tt_mask, tt_var
    for k in (4, 5):
        v = [tt_var(k, i) for i in range(k)]
        full = tt_mask(k)
        maj = (v[0] & v[1]) | (v[0] & v[2]) | (v[1] & v[2])
        f = (maj ^ v[3]) if k == 4 else ((maj & v[3]) | v[4])
        d = opt.decompose2(f, k)
        assert d is not None
        S, h_tt, T, g_tt = d
        # rebuild f from the decomposition, input by input
        h = 0
        for idx in range(1 << len(S)):
            if (h_tt >> idx) & 1:
                term = full
                for i, s in enumerate(S):
                    term &= v[s] if (idx >> i) & 1 else ~v[s] & full
                h |= term
        r = 0
        for idx in range(8):
            if (g_tt >> idx) & 1:
                ins = [h, v[T[0]], v[T[1]]]
                term = full
                for i in range(3):
                    term &= ins[i] if (idx >> i) & 1 else ~ins[i] & full
                r |= term
        assert r == f
    # the parity of four inputs is xor3(xor(a, b), c, d): g(h(a, b), c, d)
    v = [tt_var(4, i) for i in range(4)]
    assert opt.decompose2(v[0] ^ v[1] ^ v[2] ^ v[3], 4) is not None


@pytest.mark.parametrize("wE,wi,wa", [(5, 3, 4), (4, 3, 4), (5, 5, 6), (5, 10, 11)])
def test_split_asm_allocation(wE, wi, wa):
    """The register-allocated assembly of both roles computes the circuits."""
    nin, nacc = nbits(wE, wi), nbits(wE, wa)
    naccp, ninp = asmgen.pad4(nacc), asmgen.pad4(nin)
    base = asmgen.BASE
    A = list(range(base, base + naccp))
    B = list(range(base + naccp, base + 2 * naccp))
    P = list(range(base + 2 * naccp, base + 3 * naccp))
    pool = list(range(base + 3 * naccp, asmgen.TOP))
    g = np.random.default_rng([11, wE, wi, wa])
    words = 256

    def rand_words(n):
        return [g.integers(0, 2**63, words, dtype=np.uint64) * np.uint64(2) +
                g.integers(0, 2, words, dtype=np.uint64) for _ in range(n)]

    for C, ins, outs, pl in (
            (optimized("accumulate_circuit", wE, wa), {"acc": Block(A), "p": Block(P)},
             {"acc": (Block(B), "acc")}, pool),
            (optimized("product_circuit", wE, wi, wa),
             {"w": Block(range(base, base + ninp)), "x": Block(range(base + ninp, base + ninp + nin))},
             {"p": "pool"}, list(range(base + ninp + nin, asmgen.TOP)))):
        lines, place, st = regalloc.allocate(C, ins, outs, pl)
        inputs = {grp: rand_words(len(lits)) for grp, lits in C.inputs}
        want = sim.simulate(C, inputs)
        regs = {}
        for grp, _ in C.inputs:
            for r, arr in zip(place["in"][grp], inputs[grp]):
                regs[r] = arr.copy()
        for r in pl:
            regs.setdefault(r, g.integers(0, 2**63, words, dtype=np.uint64))
        regalloc.interpret(lines, regs)
        for grp, _ in C.outputs:
            for r, w in zip(place["out"][grp], want[grp]):
                assert np.array_equal(regs[r], w), (C.name, grp, r)


@pytest.mark.parametrize("K", [4, 6])
@pytest.mark.parametrize("sync", ["barrier", "pairs"])
@pytest.mark.parametrize("wE,wi,wa", [(5, 3, 4), (5, 4, 5)])
def test_split_asm_text(wE, wi, wa, sync, K):
    """Shape of the generated accumulator loop: one barrier per batch, or
    (pairs) none but a counter wait bounded by the run-time cap (a give-up
    reported) and a consumed-count store per batch; wait counts within the 4-bit field; registers within v96..v255;
    LDS offsets within the 16-bit field (a ring too deep for it is refused)."""
    import re
    nin, nacc = nbits(wE, wi), nbits(wE, wa)
    acc_c = optimized("accumulate_circuit", wE, wa)
    prod_c = optimized("product_circuit", wE, wi, wa)
    kstride = asmgen.pad4(nacc) // 4
    if (K - 1) * 4 * 64 * kstride * 16 + (kstride - 1) * 64 * 16 > 0xFFFF:
        with pytest.raises(regalloc.AllocError):
            asmgen.split_functions(acc_c, prod_c, nin, nacc, K, sync=sync)
        return
    text, _ = asmgen.split_functions(acc_c, prod_c, nin, nacc, K, sync=sync)
    offsets = [int(x) for x in re.findall(r"offset:(\d+)", text)]
    assert offsets and max(offsets) <= 0xFFFF
    loop = text[text.index("accum_loop("):text.index("kWSlot")]
    if sync == "barrier":
        assert loop.count("s_barrier") == 2
    else:
        assert "s_barrier" not in loop
        assert loop.count("s_sleep") == 2 and loop.count("v_readfirstlane_b32") == 4
        assert loop.count("ds_write_b32") == 2
        # every wait is bounded by the run-time cap, and a give-up is reported
        assert loop.count("s_cmp_ge_u32 %[spin], %[cap]") == 2
        assert loop.count("s_mov_b32 %[gave], 1") == 2 and "s_mov_b32 %[gave], 0" in loop
    waits = [int(x) for x in re.findall(r"lgkmcnt\((\d+)\)", text)]
    assert waits and max(waits) <= 15
    regs = [int(x) for x in re.findall(r"\bv(\d+)\b", text)]
    assert min(regs) >= asmgen.BASE and max(regs) < asmgen.TOP
