"""Combinational circuits as DAGs of boolean functions of at most three inputs.

This is the netlist representation of the generator. The paper builds its
operators with a hardware flow (an FP core generator, logic synthesis against a
cell library whose cells are the target's bitwise instructions, AIG
optimisation, topological sorting; Sec. 3 and the flow figure). Here the
cell library is gfx950's VALU bitwise set: every function of up to three
inputs is one instruction (``v_bitop3_b32`` takes an 8-bit truth table, like
the AVX512 ternary-logic cells of Table 1), so the natural node is a 3-input
look-up table and inverters on node inputs are free.

Signals are *literals*: ``2 * node + inverted``. Node 0 is the constant false,
so literal 0 is false and literal 1 is true. Each node stores its fan-in
nodes (sorted, distinct, each one a real dependency) and a truth table over
them, with input i weighted 2**i in the table index. Node outputs are kept in
a canonical polarity (f(0,...,0) == 0) so that complements hash together.
"""

FALSE, TRUE = 0, 1


def tt_mask(k):
    return (1 << (1 << k)) - 1


def tt_var(k, i):
    """Truth table of input i over k inputs."""
    t = 0
    for idx in range(1 << k):
        if (idx >> i) & 1:
            t |= 1 << idx
    return t


def tt_flip(tt, k, i):
    """f with input i inverted."""
    out = 0
    for idx in range(1 << k):
        if (tt >> (idx ^ (1 << i))) & 1:
            out |= 1 << idx
    return out


def tt_cofactor(tt, k, i, v):
    """f with input i fixed to v; the result is over the remaining k-1 inputs."""
    out = 0
    for j in range(1 << (k - 1)):
        lo = j & ((1 << i) - 1)
        hi = j >> i
        if (tt >> (lo | (v << i) | (hi << (i + 1)))) & 1:
            out |= 1 << j
    return out


def tt_depends(tt, k, i):
    for idx in range(1 << k):
        if ((tt >> idx) & 1) != ((tt >> (idx ^ (1 << i))) & 1):
            return True
    return False


def tt_tie(tt, k, i, j):
    """f with input j tied to input i (i < j); input j is removed."""
    out = 0
    for m in range(1 << (k - 1)):
        lo = m & ((1 << j) - 1)
        hi = m >> j
        xi = (m >> i) & 1
        if (tt >> (lo | (xi << j) | (hi << (j + 1)))) & 1:
            out |= 1 << m
    return out


def tt_permute(tt, k, perm):
    """New input p is old input perm[p]."""
    out = 0
    for idx in range(1 << k):
        old = 0
        for p in range(k):
            if (idx >> p) & 1:
                old |= 1 << perm[p]
        if (tt >> old) & 1:
            out |= 1 << idx
    return out


def normalize(tt, lits):
    """Reduce (tt, lits) to (tt, nodes) with distinct, sorted, non-constant,
    essential fan-in nodes and input inversions absorbed into tt."""
    k = len(lits)
    nodes = []
    for i, l in enumerate(lits):
        if l & 1:
            tt = tt_flip(tt, k, i)
        nodes.append(l >> 1)
    i = 0
    while i < len(nodes):  # constants (node 0 is false)
        if nodes[i] == 0:
            tt = tt_cofactor(tt, len(nodes), i, 0)
            del nodes[i]
        else:
            i += 1
    changed = True
    while changed:  # duplicated inputs
        changed = False
        for a in range(len(nodes)):
            for b in range(a + 1, len(nodes)):
                if nodes[a] == nodes[b]:
                    tt = tt_tie(tt, len(nodes), a, b)
                    del nodes[b]
                    changed = True
                    break
            if changed:
                break
    i = 0
    while i < len(nodes):  # inputs the function does not depend on
        if not tt_depends(tt, len(nodes), i):
            tt = tt_cofactor(tt, len(nodes), i, 0)
            del nodes[i]
        else:
            i += 1
    order = sorted(range(len(nodes)), key=lambda p: nodes[p])
    tt = tt_permute(tt, len(nodes), order)
    nodes = [nodes[p] for p in order]
    return tt & tt_mask(len(nodes)), nodes


class Circuit:
    """A DAG of <=3-input functions with named input and output bit-vectors."""

    def __init__(self, name):
        self.name = name
        self.fanins = [()]    # node 0: constant false
        self.tts = [0]
        self.is_input = [False]
        self.input_of = {}    # node -> (group, bit)
        self.inputs = []      # [(group, [lits])]
        self.outputs = []     # [(group, [lits])]
        self.table = {}       # (tt, fanins) -> node

    # -- construction --------------------------------------------------------
    def input(self, group, width):
        lits = []
        for b in range(width):
            n = len(self.fanins)
            self.fanins.append(())
            self.tts.append(0)
            self.is_input.append(True)
            self.input_of[n] = (group, b)
            lits.append(2 * n)
        self.inputs.append((group, lits))
        return lits

    def output(self, group, lits):
        self.outputs.append((group, list(lits)))

    def lut(self, tt, lits):
        """Literal of the function tt (input i weighted 2**i) of lits."""
        tt, nodes = normalize(tt, list(lits))
        k = len(nodes)
        if k == 0:
            return TRUE if tt & 1 else FALSE
        if k == 1 and tt in (1, 2):
            return 2 * nodes[0] + (1 if tt == 1 else 0)
        inv = tt & 1
        if inv:
            tt = ~tt & tt_mask(k)
        key = (tt, tuple(nodes))
        n = self.table.get(key)
        if n is None:
            n = len(self.fanins)
            self.fanins.append(tuple(nodes))
            self.tts.append(tt)
            self.is_input.append(False)
            self.table[key] = n
        return 2 * n + inv

    # -- gates ---------------------------------------------------------------
    @staticmethod
    def NOT(a):
        return a ^ 1

    def AND(self, a, b):
        return self.lut(0b1000, [a, b])

    def OR(self, a, b):
        return self.lut(0b1110, [a, b])

    def XOR(self, a, b):
        return self.lut(0b0110, [a, b])

    def AND3(self, a, b, c):
        return self.lut(0x80, [a, b, c])

    def OR3(self, a, b, c):
        return self.lut(0xFE, [a, b, c])

    def XOR3(self, a, b, c):
        return self.lut(0x96, [a, b, c])

    def MAJ(self, a, b, c):
        return self.lut(0xE8, [a, b, c])

    def MUX(self, s, a, b):
        """s ? a : b"""
        # inputs (s, a, b): index = s | a<<1 | b<<2
        tt = 0
        for idx in range(8):
            s_, a_, b_ = idx & 1, (idx >> 1) & 1, (idx >> 2) & 1
            if (a_ if s_ else b_):
                tt |= 1 << idx
        return self.lut(tt, [s, a, b])

    def OR_all(self, lits):
        lits = [l for l in lits if l != FALSE]
        if not lits:
            return FALSE
        while len(lits) > 1:
            nxt = []
            for i in range(0, len(lits), 3):
                grp = lits[i:i + 3]
                if len(grp) == 3:
                    nxt.append(self.OR3(*grp))
                elif len(grp) == 2:
                    nxt.append(self.OR(*grp))
                else:
                    nxt.append(grp[0])
            lits = nxt
        return lits[0]

    def AND_all(self, lits):
        return self.NOT(self.OR_all([self.NOT(l) for l in lits]))

    # -- bit-vector helpers (LSB first) ----------------------------------------
    def add(self, a, b, cin=FALSE):
        """a + b + cin over max(len) bits; returns (sum bits, carry out)."""
        n = max(len(a), len(b))
        a = list(a) + [FALSE] * (n - len(a))
        b = list(b) + [FALSE] * (n - len(b))
        s, c = [], cin
        for i in range(n):
            s.append(self.XOR3(a[i], b[i], c))
            c = self.MAJ(a[i], b[i], c)
        return s, c

    def sub(self, a, b):
        """a - b over max(len) bits (two's complement); returns (diff, borrow)."""
        n = max(len(a), len(b))
        b = list(b) + [FALSE] * (n - len(b))
        s, c = self.add(a, [self.NOT(x) for x in b], TRUE)
        return s, self.NOT(c)

    def less_than(self, a, b):
        """Unsigned a < b (the borrow of a - b)."""
        n = max(len(a), len(b))
        a = list(a) + [FALSE] * (n - len(a))
        b = list(b) + [FALSE] * (n - len(b))
        lt = FALSE
        for i in range(n):
            lt = self.MAJ(self.NOT(a[i]), b[i], lt)
        return lt

    def increment(self, a, cin):
        """a + cin; returns (bits, carry out)."""
        s, c = [], cin
        for x in a:
            s.append(self.XOR(x, c))
            c = self.AND(x, c)
        return s, c

    def mux_vec(self, s, a, b):
        return [self.MUX(s, x, y) for x, y in zip(a, b)]

    # -- queries ----------------------------------------------------------------
    def n_nodes(self):
        return sum(1 for i in range(1, len(self.fanins)) if not self.is_input[i])
