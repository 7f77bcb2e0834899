"""Emit a mapped circuit as straight-line HIP device code.

The paper's code generator turns each netlist gate into one call of a cell
function built on the target's bitwise intrinsics, one SIMD word per circuit
signal (Sec. 3.3). Here one signal is one 32-bit VGPR, i.e. the same bit of
32 independent values, and every node is one VALU instruction: three-input
nodes become ``__builtin_amdgcn_bitop3_b32`` with the node's truth table as
the immediate, two-input nodes plain C operators (which the compiler selects
as single VALU instructions) or, in an aligned function, also
``v_bitop3_b32`` (see emit_function).

``v_bitop3_b32 D, S0, S1, S2, imm`` computes, for every bit position, bit
(S0*4 + S1*2 + S2) of imm. A node's truth table weights input i by 2**i, so
the emitter passes the node's inputs as (S0, S1, S2) = (x2, x1, x0).
"""

TWO_INPUT = {0x2: "({a} & ~{b})", 0x4: "(~{a} & {b})", 0x6: "({a} ^ {b})",
             0x8: "({a} & {b})", 0xE: "({a} | {b})", 0x1: "~({a} | {b})",
             0x7: "~({a} & {b})", 0x9: "~({a} ^ {b})", 0xB: "({a} | ~{b})",
             0xD: "(~{a} | {b})"}


def schedule(C):
    """Emission order: depth-first from the outputs, larger cones first,
    so that short-lived temporaries are consumed soon after they are made."""
    size = {}

    def cone(n):
        if n in size:
            return size[n]
        if C.is_input[n] or n == 0:
            size[n] = 0
            return 0
        stack, seen = [n], set()
        while stack:
            m = stack.pop()
            if m in seen or C.is_input[m] or m == 0:
                continue
            seen.add(m)
            stack.extend(C.fanins[m])
        size[n] = len(seen)
        return size[n]

    order, done = [], set()
    for _, lits in C.outputs:
        for l in lits:
            root = l >> 1
            stack = [(root, False)]
            while stack:
                n, expanded = stack.pop()
                if n in done or n == 0 or C.is_input[n]:
                    continue
                if expanded:
                    done.add(n)
                    order.append(n)
                    continue
                stack.append((n, True))
                for f in sorted(C.fanins[n], key=cone):
                    if f not in done:
                        stack.append((f, False))
    return order


def output_polarity(C):
    """Nodes to emit complemented: those whose every use as an output is
    complemented (a LUT computes either polarity at the same cost, and LUT
    consumers absorb the flip into their truth tables)."""
    pos, neg = set(), set()
    for _, lits in C.outputs:
        for l in lits:
            n = l >> 1
            if n == 0 or C.is_input[n]:
                continue
            (neg if (l & 1) else pos).add(n)
    return neg - pos


def emit_function(C, fname, in_place=None, aligned=False):
    """C++ text of one __device__ function. Inputs are const array references
    in port order; the output group is a reference array. If in_place names an
    input group, the output overwrites that input array.

    aligned: two-input nodes also become ``v_bitop3_b32`` (with the constant 0
    as S0), so that every node is one 8-byte instruction, and the run starts
    at an 8-byte boundary (an alignment directive, then a scheduling barrier
    that keeps the nodes after it). Otherwise two-input nodes are C operators,
    which the compiler may select as 4-byte instructions."""
    from .circuit import tt_flip
    flipped = output_polarity(C)
    names = {}
    params = []
    loads = []
    for group, lits in C.inputs:
        if group == in_place:
            params.append(f"uint32_t (&{group})[{len(lits)}]")
        else:
            params.append(f"const uint32_t (&{group})[{len(lits)}]")
        for b, l in enumerate(lits):
            v = f"{group}_{b}"
            names[l >> 1] = v
            loads.append(f"  const uint32_t {v} = {group}[{b}];")
    outs = []
    for group, lits in C.outputs:
        if group != in_place:
            params.append(f"uint32_t (&{group})[{len(lits)}]")
        outs.append((group, lits))
    body = []
    for n in schedule(C):
        fan = C.fanins[n]
        k = len(fan)
        tt = C.tts[n]
        for i, f in enumerate(fan):  # fan-ins emitted complemented
            if f in flipped:
                tt = tt_flip(tt, k, i)
        if n in flipped:
            tt = ~tt & ((1 << (1 << k)) - 1)
        v = f"t{n}"
        names[n] = v
        args = [names[f] for f in fan]
        if k == 3:
            expr = f"__builtin_amdgcn_bitop3_b32({args[2]}, {args[1]}, {args[0]}, 0x{tt:02x})"
        elif k == 2 and aligned:
            expr = f"__builtin_amdgcn_bitop3_b32(0u, {args[1]}, {args[0]}, 0x{tt:02x})"
        elif k == 2:
            expr = TWO_INPUT[tt].format(a=args[0], b=args[1])
        else:
            raise ValueError(f"unexpected node arity {k}")
        body.append(f"  const uint32_t {v} = {expr};")
    stores = []
    for group, lits in outs:
        for b, l in enumerate(lits):
            n = l >> 1
            if n == 0:
                val = "0xffffffffu" if (l & 1) else "0u"
            else:
                inv = (l & 1) ^ (1 if n in flipped else 0)
                val = ("~" if inv else "") + names[n]
            stores.append(f"  {group}[{b}] = {val};")
    head = f"static __device__ __forceinline__ void {fname}({', '.join(params)})\n{{"
    # a run of 8-byte instructions issues at full rate only when it starts
    # 8-byte aligned (the assembler pads with s_nop 0)
    align = ['  asm volatile(".p2align 3");',
             "  __builtin_amdgcn_sched_barrier(0);"] if aligned else []
    return "\n".join([head] + loads + align + body + stores + ["}"]) + "\n"


def op_count(C):
    """VALU instructions the emitted function executes: one per node, plus one
    NOT per output that needs the other polarity of what its node is emitted
    in (an input copied out complemented, or a node used in both polarities)."""
    flipped = output_polarity(C)
    n = C.n_nodes()
    for _, lits in C.outputs:
        for l in lits:
            node = l >> 1
            if node != 0 and (l & 1) ^ (1 if node in flipped else 0):
                n += 1
    return n
