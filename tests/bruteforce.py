"""An independent reference for pinning the oracle (tests only).

It shares no code or structure with the oracle's rounding: values are formed
with IEEE float64 arithmetic (exact for the small formats used here, and IEEE
semantics decide NaN, infinity and zero signs), and rounding is a search for
the nearest element of the sorted list of representable values, ties going to
the element whose fraction field is even (or, toward zero, for the element of
largest magnitude not above the value's). The list spans an unbounded exponent
range around the data, so "round first, then check the exponent range" falls
out of the search.

Exactness: for wE <= 5 and wF <= 11 every product of two values has at most 24
significant bits and every sum at most 31 + 13 bits, all below float64's 53.
"""
import numpy as np


def split(codes, wE, wF):
    c = np.asarray(codes, dtype=np.uint64)
    F = (c & np.uint64((1 << wF) - 1)).astype(np.int64)
    E = ((c >> np.uint64(wF)) & np.uint64((1 << wE) - 1)).astype(np.int64)
    s = ((c >> np.uint64(wF + wE)) & np.uint64(1)).astype(np.int64)
    x = ((c >> np.uint64(wF + wE + 1)) & np.uint64(3)).astype(np.int64)
    return x, s, E, F


def to_float64(codes, wE, wF):
    """The value each code denotes, as float64 (exact for the formats here)."""
    x, s, E, F = split(codes, wE, wF)
    bias = (1 << (wE - 1)) - 1
    sign = np.where(s == 1, -1.0, 1.0)
    mag = np.ldexp((F + (1 << wF)).astype(np.float64), (E - bias - wF).astype(np.int64))
    v = np.where(x == 1, mag, np.where(x == 2, np.inf, 0.0)) * sign
    return np.where(x == 3, np.nan, v)


def _grid(wF, umin, umax):
    """All positive values (2^wF + f) * 2^(u - wF), sorted, with their (u, f)."""
    u = np.repeat(np.arange(umin, umax + 1), 1 << wF)
    f = np.tile(np.arange(1 << wF), umax - umin + 1)
    vals = np.ldexp((f + (1 << wF)).astype(np.float64), (u - wF).astype(np.int64))
    return vals, u, f


def nearest(v, wE, wF, mode="rne"):
    """Codes of float64 values v (any mix of finite, infinite, NaN, signed zero),
    rounded to nearest with ties to even fraction (mode "rne") or toward zero
    ("rtz"), then range checked."""
    v = np.asarray(v, dtype=np.float64)
    bias = (1 << (wE - 1)) - 1
    out = np.zeros(v.shape, np.uint64)
    sgn = np.signbit(v).astype(np.uint64)
    nan = np.isnan(v)
    inf = np.isinf(v)
    zero = v == 0
    fin = ~(nan | inf | zero)
    exn_shift = np.uint64(wF + wE + 1)
    s_shift = np.uint64(wF + wE)
    out[nan] = np.uint64(3) << exn_shift
    out[inf] = (np.uint64(2) << exn_shift) | (sgn[inf] << s_shift)
    out[zero] = sgn[zero] << s_shift
    if fin.any():
        a = np.abs(v[fin])
        lo_u = int(np.floor(np.log2(a.min()))) - 2
        hi_u = int(np.floor(np.log2(a.max()))) + 2
        vals, gu, gf = _grid(wF, lo_u, hi_u)
        i = np.searchsorted(vals, a, side="left")  # vals[i-1] < a <= vals[i]
        hi = vals[i]
        lo = vals[i - 1]
        d_hi = hi - a  # exact: lo and hi are within a factor two of a
        d_lo = a - lo
        if mode == "rtz":
            pick_hi = d_hi == 0
        else:
            pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (gf[i] % 2 == 0))
        j = np.where(pick_hi, i, i - 1)
        u, f = gu[j], gf[j]
        Eb = u + bias
        s = sgn[fin]
        code = (np.uint64(1) << exn_shift) | (s << s_shift) | \
            (Eb.clip(0, (1 << wE) - 1).astype(np.uint64) << np.uint64(wF)) | f.astype(np.uint64)
        code = np.where(Eb > (1 << wE) - 1, (np.uint64(2) << exn_shift) | (s << s_shift), code)
        code = np.where(Eb < 0, s << s_shift, code)
        out[fin] = code
    return out


def mul(a, b, wE, wF_in, wF_out, mode="rne"):
    return nearest(to_float64(a, wE, wF_in) * to_float64(b, wE, wF_in), wE, wF_out, mode)


def add(a, b, wE, wF, mode="rne"):
    # IEEE float64 gives +0 for x + (-x), which is this format's rule in both modes
    return nearest(to_float64(a, wE, wF) + to_float64(b, wE, wF), wE, wF, mode)


def convert(a, wE, wF_src, wF_dst, mode="rne"):
    return nearest(to_float64(a, wE, wF_src), wE, wF_dst, mode)


def relu(a, wE, wF):
    v = to_float64(a, wE, wF)
    return nearest(np.where(np.isnan(v), np.nan, np.where(v > 0, v, 0.0)), wE, wF)


def quantize(x, wE, wF):
    return nearest(np.asarray(x, dtype=np.float32).astype(np.float64), wE, wF)
