"""Format combinations the library is generated for.

Convolution variants are (wE, wF_in, wF_acc, wF_out, act): the paper's
"single" MAC types (Table 3: the multiplier and accumulator carry one more
fraction bit than the inputs) for every input mantissa width 2..10 with a
5-bit exponent (HOBFLOPS8 ... HOBFLOPS16), the IEEE-like 8-bit type
HOBFLOPSIEEE8 (4, 3), and the ReLU + format-change epilogues of a stack of
layers whose inputs alternate between (5,3) and (5,5).
Element-wise MAC variants are (wE, wF_in, wF_acc).
"""

CONV_VARIANTS = (
    [(5, m, m + 1, m + 1, 0) for m in range(2, 11)]
    + [(4, 3, 4, 4, 0)]
    + [(5, 3, 4, 5, 1), (5, 5, 6, 3, 1), (5, 3, 4, 4, 1)]
)

MULADD_VARIANTS = [(4, 2, 3), (5, 3, 4), (5, 5, 6), (5, 7, 8), (5, 10, 11), (8, 7, 8)]


def conv_tag(v):
    wE, wi, wa, wo, act = v
    return f"e{wE}m{wi}_a{wa}_o{wo}{'_relu' if act else ''}"


def muladd_tag(v):
    wE, wi, wa = v
    return f"e{wE}m{wi}_a{wa}"
