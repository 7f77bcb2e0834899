"""Bit-parallel CPU evaluation of circuits on numpy uint64 words.

Each signal is an array of uint64 words; bit j of word i is that signal in
evaluation lane 64*i + j, exactly as a bit-plane word holds one bit of 32 (on
the GPU) or 64 (here) independent values.
"""
import numpy as np

ONES = np.uint64(0xFFFFFFFFFFFFFFFF)


def _lut(tt, k, xs):
    """Evaluate a k-input truth table (input i weighted 2**i) on word arrays."""
    if k == 1:
        x = xs[0]
        return {0: np.zeros_like(x), 1: ~x, 2: x.copy(), 3: np.full_like(x, ONES)}[tt]
    if k == 2:
        a, b = xs
        return {
            0x0: np.zeros_like(a), 0x1: ~(a | b), 0x2: a & ~b, 0x3: ~b, 0x4: ~a & b, 0x5: ~a,
            0x6: a ^ b, 0x7: ~(a & b), 0x8: a & b, 0x9: ~(a ^ b), 0xA: a, 0xB: a | ~b,
            0xC: b, 0xD: ~a | b, 0xE: a | b, 0xF: np.full_like(a, ONES)}[tt]
    # Shannon expansion on the last input
    lo, hi = tt & 0xF, tt >> 4
    c = xs[2]
    f0 = _lut(lo, 2, xs[:2])
    f1 = _lut(hi, 2, xs[:2])
    return (c & f1) | (~c & f0)


def simulate(C, inputs):
    """inputs: {group: [word array per bit]} -> {group: [word array per bit]}."""
    val = {}
    for group, lits in C.inputs:
        arrs = inputs[group]
        assert len(arrs) == len(lits)
        for l, arr in zip(lits, arrs):
            val[l >> 1] = np.asarray(arr, dtype=np.uint64)
    shape = next(iter(val.values())).shape
    zero = np.zeros(shape, np.uint64)
    # reference counts, so that dead values are freed early
    needed = set()
    stack = [l >> 1 for _, lits in C.outputs for l in lits]
    while stack:
        n = stack.pop()
        if n in needed or n == 0:
            continue
        needed.add(n)
        stack.extend(C.fanins[n])
    uses = {}
    for n in needed:
        for f in C.fanins[n]:
            uses[f] = uses.get(f, 0) + 1
    for _, lits in C.outputs:
        for l in lits:
            uses[l >> 1] = uses.get(l >> 1, 0) + 1
    for n in sorted(needed):
        if C.is_input[n]:
            continue
        fan = C.fanins[n]
        val[n] = _lut(C.tts[n], len(fan), [val[f] for f in fan])
        for f in fan:
            uses[f] -= 1
            if uses[f] == 0 and not C.is_input[f]:
                del val[f]
    out = {}
    for group, lits in C.outputs:
        arrs = []
        for l in lits:
            v = zero if (l >> 1) == 0 else val[l >> 1]
            arrs.append(~v if (l & 1) else v.copy())
        out[group] = arrs
    return out


# -- conversion between codes and bit-planes ------------------------------------

def codes_to_planes(codes, nbits):
    """uint codes (n values, n a multiple of 64) -> list of nbits word arrays."""
    c = np.asarray(codes, dtype=np.uint64)
    assert c.size % 64 == 0
    planes = []
    for b in range(nbits):
        bits = ((c >> np.uint64(b)) & np.uint64(1)).astype(np.uint8)
        packed = np.packbits(bits.reshape(-1, 64), axis=1, bitorder="little")
        planes.append(packed.view(np.uint64).reshape(-1))
    return planes


def planes_to_codes(planes):
    out = None
    for b, p in enumerate(planes):
        bits = np.unpackbits(np.asarray(p, np.uint64).view(np.uint8), bitorder="little")
        v = bits.astype(np.uint64) << np.uint64(b)
        out = v if out is None else (out | v)
    return out


def exhaustive_planes(nbits):
    """Planes enumerating all 2**nbits input patterns (pattern index = lane)."""
    n = 1 << nbits
    words = max(n // 64, 1)
    idx = np.arange(words, dtype=np.uint64)
    planes = []
    lane_pat = [0xAAAAAAAAAAAAAAAA, 0xCCCCCCCCCCCCCCCC, 0xF0F0F0F0F0F0F0F0,
                0xFF00FF00FF00FF00, 0xFFFF0000FFFF0000, 0xFFFFFFFF00000000]
    for b in range(nbits):
        if b < 6:
            planes.append(np.full(words, np.uint64(lane_pat[b]), np.uint64))
        else:
            planes.append(np.where((idx >> np.uint64(b - 6)) & np.uint64(1), ONES,
                                   np.uint64(0)).astype(np.uint64))
    return planes
