"""Format combinations and rounding modes the library is generated for.

Convolution variants are (wE, wF_in, wF_acc, wF_out, act, round):
  * the paper's type sweep (Table 3): HOBFLOPS8 ... HOBFLOPS16, inputs (5, m)
    for m = 2..10, and HOBFLOPSIEEE8, inputs (4, 3); each as the "single" MAC
    type (multiplier and accumulator carry wF+1 fraction bits) and as the
    "extended" type (2wF+1 bits: the product is exact), each rounding to
    nearest even and toward zero (Sec. 4);
  * the ReLU + format-change epilogues of a stack of layers whose inputs
    alternate between (5,3) and (5,5);
  * HOBFLOPS9 accumulating in its own input format, (5,3) -> (5,3): the
    small convolution read literally, "accumulate in the same format".
Element-wise MAC variants are (wE, wF_in, wF_acc, round).
Global average pooling variants are (wE, wF_in, wF_acc, wF_out, round): the
output format of every "single" convolution variant of the sweep pooled in
that format, and (5,4) pooled with one more fraction bit in the sum.
"""
RNE, RTZ = 0, 1

SWEEP_TYPES = [(5, m) for m in range(2, 11)] + [(4, 3)]

CONV_VARIANTS = (
    [(wE, m, m + 1, m + 1, 0, r) for r in (RNE, RTZ) for wE, m in SWEEP_TYPES]
    + [(wE, m, 2 * m + 1, 2 * m + 1, 0, r) for r in (RNE, RTZ) for wE, m in SWEEP_TYPES]
    + [(5, 3, 4, 5, 1, RNE), (5, 5, 6, 3, 1, RNE), (5, 3, 4, 4, 1, RNE)]
    + [(5, 3, 3, 3, 0, r) for r in (RNE, RTZ)]
)

MULADD_VARIANTS = [(wE, wi, wa, r) for r in (RNE, RTZ) for wE, wi, wa in
                   [(4, 2, 3), (5, 3, 4), (5, 5, 6), (5, 7, 8), (5, 10, 11), (8, 7, 8)]]

POOL_VARIANTS = (
    [(wE, m + 1, m + 1, m + 1, r) for r in (RNE, RTZ) for wE, m in SWEEP_TYPES]
    + [(5, 4, 5, 4, RNE), (5, 4, 5, 4, RTZ)]
)

RND_NAME = {RNE: "rne", RTZ: "rtz"}


def _sfx(r):
    return "" if r == RNE else "_" + RND_NAME[r]


def conv_tag(v):
    wE, wi, wa, wo, act, r = v
    return f"e{wE}m{wi}_a{wa}_o{wo}{'_relu' if act else ''}{_sfx(r)}"


def muladd_tag(v):
    wE, wi, wa, r = v
    return f"e{wE}m{wi}_a{wa}{_sfx(r)}"


def pool_tag(v):
    wE, wi, wa, wo, r = v
    return f"e{wE}m{wi}_a{wa}_o{wo}{_sfx(r)}"
