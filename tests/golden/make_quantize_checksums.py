"""Writes quantize_all_f32.json: per chunk of 2^28 consecutive float32 bit
patterns (all 2^32 of them in 16 chunks), a checksum of the oracle's codes
for every pattern, for the formats listed. Calls only oracle/ (quantisation
of float32 to a (wE, wF) code, paper Sec. 3.1 and 3.3 with rounding to
nearest even, Sec. 4). Run from the repository root:

    python tests/golden/make_quantize_checksums.py

The checksum of a chunk is sum over its patterns i of ((code + 1) * h(i))
mod P, with h(i) = (A * (i mod P) + B) mod P, for two (A, B, P) triples; all
intermediate values stay below 2^63, so numpy and torch int64 compute it
exactly. A code that differs changes a checksum unless two errors cancel.
"""
import json
import os
import sys
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

CHUNK_BITS = 28
HASHES = [(1103515245, 12345, 2147483629), (69069, 1, 2147483587)]  # (A, B, P), P prime
# (5,3): the bench's input format, rounded by the add-and-subtract quantiser
# of the pack kernel; (8,7): eight exponent bits, the integer quantiser;
# (6,23): every fraction bit kept (nothing to round); (2,1): the narrowest
FORMATS = [(5, 3), (8, 7), (6, 23), (2, 1)]
SUB = 1 << 22


def checksum_terms(codes, first, A, B, P):
    i = np.arange(first, first + codes.size, dtype=np.int64)
    h = (A * (i % P) + B) % P
    return int((((codes.astype(np.int64) + 1) % P) * h % P).sum() % P)


def chunk_checksums(args):
    wE, wF, c = args
    import oracle
    sums = [0] * len(HASHES)
    base = c << CHUNK_BITS
    for s in range(0, 1 << CHUNK_BITS, SUB):
        bits = np.arange(base + s, base + s + SUB, dtype=np.uint64).astype(np.uint32)
        codes = oracle.quantize_f32(bits.view(np.float32), wE, wF).astype(np.int64)
        for k, (A, B, P) in enumerate(HASHES):
            sums[k] = (sums[k] + checksum_terms(codes, base + s, A, B, P)) % P
    return sums


def main():
    path = os.path.join(HERE, "quantize_all_f32.json")
    out = {"source": "oracle.quantize_f32 over every float32 bit pattern, written by "
                     "tests/golden/make_quantize_checksums.py (calls only oracle/)",
           "chunk_bits": CHUNK_BITS, "hashes": HASHES, "formats": {}}
    if os.path.exists(path):  # formats already there are kept (an hour of CPU each)
        old = json.load(open(path))
        if old["chunk_bits"] == CHUNK_BITS and old["hashes"] == [list(h) for h in HASHES]:
            out["formats"] = old["formats"]
    with ProcessPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        for wE, wF in FORMATS:
            if f"{wE},{wF}" in out["formats"]:
                continue
            chunks = list(ex.map(chunk_checksums,
                                 [(wE, wF, c) for c in range(1 << (32 - CHUNK_BITS))]))
            out["formats"][f"{wE},{wF}"] = chunks
            print(wE, wF, "done", flush=True)
            with open(path, "w") as f:
                json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
