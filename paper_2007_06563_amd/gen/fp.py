"""Bit-level floating-point operator circuits in the FloPoCo word format.

A value of format (wE, wF) is NB = 3 + wE + wF signals, LSB first: fraction
F (wF), exponent E (wE), sign s, exception field x0 (LSB) and x1 (MSB). The
exception field is 00 zero, 01 normal, 10 infinity, 11 NaN (paper Sec. 3.3
defines 01 as normal and the format as having no subnormals; the other three
codes follow FloPoCo, the generator the paper uses). The exponent bias is
2^(wE-1) - 1 and every exponent value is an ordinary binade.

The operators compute what the paper's multiplier and adder compute: an exact
result rounded to nearest, ties to even (Sec. 4), with the exponent range
checked after rounding (overflow to infinity, underflow to a signed zero),
IEEE-754 rules for NaN, infinity and zero signs (Sec. 3.3 notes the operators
match IEEE-754 on quantized values), and a multiplier whose output may have
more fraction bits than its inputs (Table 3).

With ``canonical=False`` an operator may leave arbitrary E and F bits on a
non-normal result and an arbitrary sign on NaN. Every operator here reads only
(x, s) of non-normal inputs, so such values are safe between operators; the
last operator before a result leaves the GPU must be canonical.
"""
from .circuit import FALSE, TRUE, Circuit


class FP:
    def __init__(self, lits, wE, wF):
        assert len(lits) == 3 + wE + wF
        self.wE, self.wF = wE, wF
        self.F = list(lits[:wF])
        self.E = list(lits[wF:wF + wE])
        self.s = lits[wF + wE]
        self.x0 = lits[wF + wE + 1]
        self.x1 = lits[wF + wE + 2]


def nb(wE, wF):
    return 3 + wE + wF


def classify(C: Circuit, v: FP):
    """(nan, inf, zero, normal) flags of a value."""
    n = C.NOT
    return (C.AND(v.x1, v.x0), C.AND(v.x1, n(v.x0)), C.AND(n(v.x1), n(v.x0)),
            C.AND(n(v.x1), v.x0))


def assemble(C: Circuit, F, E, s, is_nan, is_inf, is_norm, canonical):
    x1 = C.OR(is_nan, is_inf)
    x0 = C.OR(is_nan, is_norm)
    if canonical:
        F = [C.AND(f, is_norm) for f in F]
        E = [C.AND(e, is_norm) for e in E]
        s = C.AND(s, C.NOT(is_nan))
    return list(F) + list(E) + [s, x0, x1]


def multiply_unsigned(C: Circuit, a, b):
    """Exact product of two unsigned bit-vectors: partial products reduced by
    full adders column by column, then one ripple-carry adder."""
    cols = [[] for _ in range(len(a) + len(b))]
    for i, x in enumerate(a):
        for j, y in enumerate(b):
            p = C.AND(x, y)
            if p != FALSE:
                cols[i + j].append(p)
    while max(len(c) for c in cols) > 2:
        new = [[] for _ in range(len(cols) + 1)]
        for k, col in enumerate(cols):
            i = 0
            while len(col) - i >= 3:
                x, y, z = col[i:i + 3]
                i += 3
                new[k].append(C.XOR3(x, y, z))
                new[k + 1].append(C.MAJ(x, y, z))
            new[k].extend(col[i:])
        assert not new[len(cols)], "product overflowed its width"
        cols = new[:len(cols)]
    out, c = [], FALSE
    for col in cols:
        x = col[0] if col else FALSE
        y = col[1] if len(col) > 1 else FALSE
        out.append(C.XOR3(x, y, c))
        c = C.MAJ(x, y, c)
    return out


def signed_const(value, width):
    return [TRUE if (value >> i) & 1 else FALSE for i in range(width)]


def fp_mul(C: Circuit, A, B, wE, wF, wFo, canonical=True, rnd="rne"):
    """(wE, wF) x (wE, wF) -> (wE, wFo), rounded once: to nearest, ties to
    even ("rne"), or toward zero ("rtz": the dropped bits are discarded)."""
    a, b = FP(A, wE, wF), FP(B, wE, wF)
    nan_a, inf_a, zero_a, norm_a = classify(C, a)
    nan_b, inf_b, zero_b, norm_b = classify(C, b)
    s = C.XOR(a.s, b.s)

    P = multiply_unsigned(C, a.F + [TRUE], b.F + [TRUE])  # 2wF+2 bits
    top = 2 * wF + 1
    n = P[top]  # product >= 2: the leading one is one place higher

    def bit(i):
        return P[i] if 0 <= i < len(P) else FALSE

    frac = [C.MUX(n, bit(top - wFo + i), bit(top - 1 - wFo + i)) for i in range(wFo)]
    rb = C.MUX(n, bit(top - 1 - wFo), bit(top - 2 - wFo))
    st = C.OR(C.OR_all([bit(i) for i in range(0, top - 2 - wFo)]),
              C.AND(n, bit(top - 2 - wFo)))
    round_up = C.AND(rb, C.OR(st, frac[0])) if rnd == "rne" else FALSE
    frac, rc = C.increment(frac, round_up)

    # exponent Ea + Eb - bias + n + rc in (wE+2)-bit two's complement
    bias = (1 << (wE - 1)) - 1
    if wFo >= wF:
        # n and rc are never both set: with n the kept bits cannot all be ones
        S, c = C.add(a.E, b.E, C.OR(n, rc))
        T, _ = C.add(S + [c, FALSE], signed_const(-bias, wE + 2), FALSE)
    else:
        S, c = C.add(a.E, b.E, n)
        T, _ = C.add(S + [c, FALSE], signed_const(-bias, wE + 2), rc)
    neg = T[wE + 1]
    ovf = C.AND(C.NOT(neg), T[wE])
    unf = neg

    both = C.AND(norm_a, norm_b)
    # an operand's x1 (infinity or NaN) stands in for "infinity": they differ
    # only where a NaN operand already makes the result NaN
    nan = C.OR(C.OR(nan_a, nan_b), C.OR(C.AND(a.x1, zero_b), C.AND(zero_a, b.x1)))
    inf = C.AND(C.NOT(nan), C.OR(C.OR(a.x1, b.x1), C.AND(both, ovf)))
    is_norm = C.AND(both, C.NOT(C.OR(ovf, unf)))
    return assemble(C, frac, T[:wE], s, nan, inf, is_norm, canonical)


def fp_add(C: Circuit, A, B, wE, wF, canonical=True, rnd="rne", late_clear=True,
           diff_mux=False):
    """(wE, wF) + (wE, wF) -> (wE, wF), rounded once ("rne" or "rtz"; with
    the sticky bit as the sum's least significant bit, truncating the computed
    sum truncates the exact one). late_clear and diff_mux pick between
    equivalent structures of the alignment (below); the optimiser maps each a
    little differently."""
    a, b = FP(A, wE, wF), FP(B, wE, wF)
    nan_a, inf_a, zero_a, norm_a = classify(C, a)
    nan_b, inf_b, zero_b, norm_b = classify(C, b)
    NOT = C.NOT

    # Order by magnitude on the key (x0, E, F): a zero operand (x0 = 0) is
    # always the smaller one; infinities and NaNs are decided further down.
    sw = C.less_than(a.F + a.E + [a.x0], b.F + b.E + [b.x0])
    XE, YE = C.mux_vec(sw, b.E, a.E), C.mux_vec(sw, a.E, b.E)
    XF, YF = C.mux_vec(sw, b.F, a.F), C.mux_vec(sw, a.F, b.F)
    sX = C.MUX(sw, b.s, a.s)
    nY = C.MUX(sw, a.x0, b.x0)  # the smaller operand is normal (else zero)
    eff = C.XOR(a.s, b.s)       # effective subtraction

    # Align the smaller significand: window positions 0..wF+2 hold guard and
    # round below it; everything shifted further right is ORed into sticky.
    # The window is cleared when the smaller operand is zero or shifted out
    # whole: either before the shift (late_clear False) or after it, which
    # gives the same window and sticky bit.
    if diff_mux:  # XE - YE as one of the two differences of the unswapped exponents
        d = C.mux_vec(sw, C.sub(b.E, a.E)[0], C.sub(a.E, b.E)[0])
    else:
        d, _ = C.sub(XE, YE)
    nst = (wF + 2).bit_length()
    big = C.OR_all(d[nst:]) if wE > nst else FALSE
    keep = C.AND(nY, NOT(big))
    if late_clear:
        win = [FALSE, FALSE] + list(YF) + [TRUE]
        st = FALSE
    else:
        win = [FALSE, FALSE] + [C.AND(f, keep) for f in YF] + [keep]
        st = C.AND(nY, big)
    for k in range(min(nst, wE)):
        sh = 1 << k
        gone = C.OR_all(win[:sh])
        st = C.OR(st, C.AND(d[k], gone))
        win = [C.MUX(d[k], win[p + sh] if p + sh < len(win) else FALSE, win[p])
               for p in range(len(win))]
    if late_clear:
        win = [C.AND(w, keep) for w in win]
        st = C.OR(C.AND(st, keep), C.AND(nY, big))

    # Add or subtract, sticky as the least significant bit.
    xv = [FALSE, FALSE, FALSE] + XF + [TRUE]
    yv = [st] + win
    r, c = [], eff
    for i in range(len(xv)):
        yi = C.XOR(yv[i], eff)
        r.append(C.XOR3(xv[i], yi, c))
        c = C.MAJ(xv[i], yi, c)
    r.append(C.AND(c, NOT(eff)))  # carry out counts only for an addition
    W = len(r)                    # wF + 5

    # Normalise: shift the leading one to the top, largest step first.
    nrm = (wF + 2).bit_length()
    L = [None] * nrm
    v = r
    for k in reversed(range(nrm)):
        sh = 1 << k
        z = NOT(C.OR_all(v[W - sh:]))
        L[k] = z
        v = [C.MUX(z, v[p - sh] if p >= sh else FALSE, v[p]) for p in range(W)]
    nonzero = v[W - 1]

    # Round to nearest even.
    frac = v[W - 1 - wF:W - 1]
    rb = v[W - 2 - wF]
    stk = C.OR_all(v[:W - 2 - wF])
    round_up = C.AND(rb, C.OR(stk, frac[0])) if rnd == "rne" else FALSE
    frac, rc = C.increment(frac, round_up)

    # Exponent XE + 1 - L + rc in (wE+2)-bit two's complement.
    K, _ = C.sub(signed_const(1, wE + 2), L + [FALSE] * (wE + 2 - nrm))
    T, _ = C.add(XE + [FALSE, FALSE], K, rc)
    neg = T[wE + 1]
    ovf = C.AND(NOT(neg), T[wE])
    unf = neg

    dp = C.AND(NOT(a.x1), NOT(b.x1))   # no infinity or NaN operand
    both_zero = C.AND(NOT(a.x0), NOT(b.x0))
    dpv = C.AND(dp, NOT(both_zero))    # the datapath result stands
    # A NaN operand makes the result NaN whatever else holds, so below an
    # operand's x1 (infinity or NaN) stands in for "infinity": the two differ
    # only where the result is NaN, whose sign is not read (and is cleared in
    # canonical form).
    nan = C.OR(C.OR(nan_a, nan_b), C.AND(C.AND(a.x1, b.x1), eff))
    inf = C.AND(NOT(nan), C.OR(C.OR(a.x1, b.x1), C.AND(C.AND(dpv, nonzero), ovf)))
    is_norm = C.AND(C.AND(dpv, nonzero), NOT(C.OR(ovf, unf)))
    # zero results: both zero -> -0 only if both -0; cancellation -> +0;
    # underflow -> sign of the exact value
    s_dp = C.MUX(both_zero, C.AND(a.s, b.s), C.AND(nonzero, sX))
    s = C.MUX(C.OR(a.x1, b.x1), C.MUX(a.x1, a.s, b.s), s_dp)
    return assemble(C, frac, T[:wE], s, nan, inf, is_norm, canonical)


def fp_convert(C: Circuit, A, wE, wFs, wFd, relu=False, canonical=True, rnd="rne"):
    """(wE, wFs) -> (wE, wFd): exact widening or narrowing rounded to nearest
    even ("rne") or toward zero ("rtz"), with an optional ReLU first (NaN
    stays NaN; any negative value or -0 becomes +0)."""
    a = FP(A, wE, wFs)
    nan, inf, zero, norm = classify(C, a)
    if wFd >= wFs:
        F = [FALSE] * (wFd - wFs) + a.F
        E = a.E
        ovf = FALSE
    else:
        D = wFs - wFd
        rb = a.F[D - 1]
        st = C.OR_all(a.F[:D - 1])
        kept = a.F[D:]
        round_up = C.AND(rb, C.OR(st, kept[0] if kept else TRUE)) if rnd == "rne" else FALSE
        F, c = C.increment(kept, round_up)
        E, ovf = C.increment(a.E, c)
    s = a.s
    is_inf = C.OR(inf, C.AND(norm, ovf))
    is_norm = C.AND(norm, C.NOT(ovf))
    if relu:
        kill = C.AND(s, C.NOT(nan))
        is_inf = C.AND(is_inf, C.NOT(kill))
        is_norm = C.AND(is_norm, C.NOT(kill))
        s = C.AND(s, C.NOT(kill))
    return assemble(C, F, E, s, nan, is_inf, is_norm, canonical)


# ---------------------------------------------------------------------------
# Whole circuits with named ports.

def _sfx(rnd):
    return "" if rnd == "rne" else "_" + rnd


def mul_circuit(wE, wF, wFo, canonical=True, rnd="rne"):
    C = Circuit(f"mul_e{wE}m{wF}_m{wFo}{_sfx(rnd)}")
    a = C.input("a", nb(wE, wF))
    b = C.input("b", nb(wE, wF))
    C.output("r", fp_mul(C, a, b, wE, wF, wFo, canonical, rnd))
    return C


def add_circuit(wE, wF, canonical=True, rnd="rne"):
    C = Circuit(f"add_e{wE}m{wF}{_sfx(rnd)}")
    a = C.input("a", nb(wE, wF))
    b = C.input("b", nb(wE, wF))
    C.output("r", fp_add(C, a, b, wE, wF, canonical, rnd))
    return C


def convert_circuit(wE, wFs, wFd, relu=False, canonical=True, rnd="rne"):
    C = Circuit(f"cvt_e{wE}m{wFs}_m{wFd}{'_relu' if relu else ''}{_sfx(rnd)}")
    a = C.input("a", nb(wE, wFs))
    C.output("r", fp_convert(C, a, wE, wFs, wFd, relu, canonical, rnd))
    return C


def widen(lits, wE, wFs, wFd):
    """Exact widening of the fraction: no gates, only wiring."""
    v = FP(lits, wE, wFs)
    return [FALSE] * (wFd - wFs) + v.F + v.E + [v.s, v.x0, v.x1]


def muladd_circuit(wE, wF, wFacc, rnd="rne"):
    """r = add(widen(c), mul(a, b)) in (wE, wFacc): the element-wise MAC."""
    C = Circuit(f"muladd_e{wE}m{wF}_m{wFacc}{_sfx(rnd)}")
    a = C.input("a", nb(wE, wF))
    b = C.input("b", nb(wE, wF))
    c = C.input("c", nb(wE, wF))
    p = fp_mul(C, a, b, wE, wF, wFacc, canonical=False, rnd=rnd)
    C.output("r", fp_add(C, widen(c, wE, wF, wFacc), p, wE, wFacc, canonical=True, rnd=rnd))
    return C


def product_circuit(wE, wF, wFacc, rnd="rne"):
    """p = mul(w, x) for the convolution, non-canonical (feeds only the adder)."""
    C = Circuit(f"prod_e{wE}m{wF}_m{wFacc}{_sfx(rnd)}")
    w = C.input("w", nb(wE, wF))
    x = C.input("x", nb(wE, wF))
    C.output("p", fp_mul(C, w, x, wE, wF, wFacc, canonical=False, rnd=rnd))
    return C


def accumulate_circuit(wE, wFacc, rnd="rne", late_clear=True, diff_mux=True):
    """acc' = add(acc, p) for the convolution, non-canonical in and out."""
    C = Circuit(f"accum_e{wE}m{wFacc}{_sfx(rnd)}")
    acc = C.input("acc", nb(wE, wFacc))
    p = C.input("p", nb(wE, wFacc))
    C.output("acc", fp_add(C, acc, p, wE, wFacc, canonical=False, rnd=rnd,
                           late_clear=late_clear, diff_mux=diff_mux))
    return C


def mac_circuit(wE, wF, wFacc, rnd="rne"):
    """acc' = add(acc, mul(w, x)): one step of the convolution's accumulation.
    Intermediate accumulators need not be canonical."""
    C = Circuit(f"mac_e{wE}m{wF}_m{wFacc}{_sfx(rnd)}")
    acc = C.input("acc", nb(wE, wFacc))
    w = C.input("w", nb(wE, wF))
    x = C.input("x", nb(wE, wF))
    p = fp_mul(C, w, x, wE, wF, wFacc, canonical=False, rnd=rnd)
    C.output("acc", fp_add(C, acc, p, wE, wFacc, canonical=False, rnd=rnd))
    return C
