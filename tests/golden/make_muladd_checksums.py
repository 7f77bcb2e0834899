"""Writes muladd_all_codes.json: for small formats, every triple of codes
(a, b, c) -- 2^(3 NB) of them, non-canonical specials included -- through
oracle.muladd (add(widen(c), mul(a, b)), each rounded, paper Sec. 3.3 and
Table 3; nearest even or toward zero, Sec. 4), and per chunk of 2^24 triples
two modular checksums of the result codes. Triple i has a = i mod 2^NB,
b = (i >> NB) mod 2^NB, c = i >> 2 NB. Calls only oracle/. Run from the
repository root:

    python tests/golden/make_muladd_checksums.py

The checksum is the one of make_quantize_checksums.py.
"""
import json
import os
import sys
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

from make_quantize_checksums import HASHES, checksum_terms  # noqa: E402

CHUNK_BITS = 24
# (wE, wF_in, wF_acc, rounding): the generated element-wise variants with at
# most 11 bits a code, (4,2) and HOBFLOPS9's (5,3), both roundings
CASES = [(4, 2, 3, "rne"), (4, 2, 3, "rtz"), (5, 3, 4, "rne"), (5, 3, 4, "rtz")]
SUB = 1 << 21


def chunk_checksums(args):
    wE, wi, wa, rnd, c = args
    import oracle
    nb = 3 + wE + wi
    mask = (1 << nb) - 1
    sums = [0] * len(HASHES)
    base = c << CHUNK_BITS
    for s in range(0, 1 << CHUNK_BITS, SUB):
        i = np.arange(base + s, base + s + SUB, dtype=np.uint64)
        a, b, cc = i & np.uint64(mask), (i >> np.uint64(nb)) & np.uint64(mask), i >> np.uint64(2 * nb)
        r = oracle.muladd(a, b, cc, wE, wi, wa, rnd=oracle.RNE if rnd == "rne" else oracle.RTZ)
        for k, (A, B, P) in enumerate(HASHES):
            sums[k] = (sums[k] + checksum_terms(r.astype(np.int64), base + s, A, B, P)) % P
    return sums


def main():
    out = {"source": "oracle.muladd over every triple of codes, written by "
                     "tests/golden/make_muladd_checksums.py (calls only oracle/)",
           "chunk_bits": CHUNK_BITS, "hashes": HASHES, "cases": {}}
    with ProcessPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        for wE, wi, wa, rnd in CASES:
            nchunks = 1 << max(0, 3 * (3 + wE + wi) - CHUNK_BITS)
            out["cases"][f"{wE},{wi},{wa},{rnd}"] = list(
                ex.map(chunk_checksums, [(wE, wi, wa, rnd, c) for c in range(nchunks)]))
            print(wE, wi, wa, rnd, "done", flush=True)
    with open(os.path.join(HERE, "muladd_all_codes.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
