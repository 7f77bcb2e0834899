"""PL32 layout in numpy (tests only): codes [rows, len] <-> words [rows, G, NB].

Bit j of words[r, g, b] is bit b of the code of element (r, 32g + j); lanes
past len are zero. Layout only -- no arithmetic of the number format.
"""
import numpy as np


def pack_codes(codes, nbits):
    c = np.asarray(codes, dtype=np.uint64)
    rows, length = c.shape
    G = (length + 31) // 32
    padded = np.zeros((rows, G * 32), np.uint64)
    padded[:, :length] = c
    padded = padded.reshape(rows, G, 32)
    out = np.zeros((rows, G, nbits), np.uint32)
    for b in range(nbits):
        bits = ((padded >> np.uint64(b)) & np.uint64(1)).astype(np.uint64)
        out[:, :, b] = (bits << np.arange(32, dtype=np.uint64)).sum(axis=2).astype(np.uint32)
    return out


def unpack_planes(words, length):
    w = np.asarray(words).view(np.uint32) if np.asarray(words).dtype == np.int32 else \
        np.asarray(words, dtype=np.uint32)
    rows, G, nbits = w.shape
    lanes = np.arange(32, dtype=np.uint32)
    codes = np.zeros((rows, G, 32), np.uint64)
    for b in range(nbits):
        bit = (w[:, :, b][:, :, None] >> lanes) & np.uint32(1)
        codes |= bit.astype(np.uint64) << np.uint64(b)
    return codes.reshape(rows, G * 32)[:, :length]
