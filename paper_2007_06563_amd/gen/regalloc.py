"""Bank-aware register allocation and gfx950 assembly for mapped netlists.

A VGPR of gfx950 lives in bank (register number mod 4). With two or more waves
on a SIMD, a VALU instruction whose source VGPRs share a bank issues at about
two thirds of the rate (measured on MI355X with straight-line v_bitop3_b32 and
the cycle counter: 2.25 clocks per instruction per SIMD with three distinct
banks, 3.3 with two or three sources in one bank; one wave alone issues every
~4.5 clocks either way). The compiler's register allocator does not look at
banks, so the netlists are emitted here as assembly with explicit registers:

* every value (port bit, LUT node) gets a bank so that the sources of each
  instruction are in pairwise distinct banks: greedy colouring of the
  "read together" graph, most-constrained value first. A port whose bits sit
  in a block of registers (filled by 16-byte LDS loads) may put any bit in any
  register of the block, so its bits get banks within the block's capacity
  per bank, and the caller learns the resulting bit -> register permutation;
* registers are then assigned by a linear scan over the emission order, per
  bank, from a pool of temporaries;
* three-input nodes become ``v_bitop3_b32`` (operands x2, x1, x0 so that the
  node's truth table is the immediate); two-input nodes become
  ``v_bitop3_b32`` with an inline-constant third operand, so they read two
  VGPRs only.

``interpret`` executes the produced instruction list on numpy words, for
checking the allocation against the circuit on the CPU.
"""
from collections import defaultdict

import numpy as np

from .circuit import tt_flip
from .emit import output_polarity, schedule

NBANK = 4


def bank(reg):
    return reg % NBANK


class AllocError(RuntimeError):
    pass


class Block:
    """A set of registers a port's bits may be placed in, one bit per register."""

    def __init__(self, regs):
        self.regs = list(regs)

    def capacity(self):
        cap = [0] * NBANK
        for r in self.regs:
            cap[bank(r)] += 1
        return cap


def list_schedule(C, gap=2):
    """Emission order for straight-line asm: a ready node is preferred when it
    does not read a result of the last `gap` instructions, then when it frees
    more registers than it defines, then by the length of the longest path
    below it. (On MI355X a dependent instruction right after its producer
    measured no slower; the spacing costs nothing and keeps the order robust
    to a deeper pipeline.)"""
    live_nodes = set()
    stack = [l >> 1 for _, lits in C.outputs for l in lits]
    while stack:
        n = stack.pop()
        if n in live_nodes or n == 0 or C.is_input[n]:
            continue
        live_nodes.add(n)
        stack.extend(C.fanins[n])
    users = defaultdict(list)
    for n in live_nodes:
        for f in C.fanins[n]:
            users[f].append(n)
    height = {}
    for n in sorted(live_nodes, reverse=True):  # node ids are topological
        height[n] = 1 + max((height[u] for u in users[n]), default=0)
    out_use = defaultdict(int)
    for _, lits in C.outputs:
        for l in lits:
            out_use[l >> 1] += 1
    remaining = {f: len(us) for f, us in users.items()}
    waiting = {n: sum(1 for f in C.fanins[n] if f in live_nodes) for n in live_nodes}
    ready = set(n for n in live_nodes if waiting[n] == 0)
    order, recent = [], []
    while ready:
        def key(n):
            dep = any(f in recent for f in C.fanins[n])
            frees = sum(1 for f in C.fanins[n] if remaining[f] == 1 and out_use[f] == 0)
            return (not dep, frees - 1, height[n], -n)
        n = max(ready, key=key)
        ready.discard(n)
        order.append(n)
        recent = (recent + [n])[-gap:]
        for f in C.fanins[n]:
            remaining[f] -= 1
        for u in users[n]:
            waiting[u] -= 1
            if waiting[u] == 0:
                ready.add(u)
    assert len(order) == len(live_nodes)
    return order


def allocate(C, in_ports, out_ports, pool, order=None):
    """Assembly for circuit C.

    in_ports:  {group: list of registers | Block}
    out_ports: {group: list of registers | (Block, tied input group) | "pool"};
               a tied output bit b goes to the register of its block at the
               same index as input bit b of the tied group in that group's
               block, so the two blocks must have the same bank pattern; a
               "pool" output stays in whatever temporary holds it at the end.
    pool:      registers for temporaries (disjoint from all port registers).
    Returns (lines, placement, stats): placement["in"][group] and
    placement["out"][group] list the register of every bit of every port.
    """
    order = order or list_schedule(C)
    flipped = output_polarity(C)
    groups_in = dict(C.inputs)
    groups_out = dict(C.outputs)

    # ---- values, their uses, lifetimes
    nodes = list(order)
    pos = {n: i for i, n in enumerate(nodes)}
    end = len(nodes)
    last = {}
    for i, n in enumerate(nodes):
        for f in C.fanins[n]:
            last[f] = i

    # output bits: node emitted straight into the output register when it is
    # needed there in its emitted polarity and not already claimed
    out_direct = {}      # node -> (group, bit)
    copies = []          # (group, bit, kind, src node, invert)
    for group, lits in C.outputs:
        for b, l in enumerate(lits):
            n = l >> 1
            if n == 0:
                copies.append((group, b, "const", 0xFFFFFFFF if (l & 1) else 0, 0))
                continue
            inv = (l & 1) ^ (1 if n in flipped else 0)
            if out_ports[group] == "pool":
                if not C.is_input[n] and not inv:
                    last[n] = end      # stays live in its temporary
                else:
                    copies.append((group, b, "copy", n, inv))
                    last[n] = end
            elif not C.is_input[n] and not inv and n not in out_direct:
                out_direct[n] = (group, b)
            else:
                copies.append((group, b, "copy", n, inv))
                last[n] = end
    for n in out_direct:
        last[n] = max(last.get(n, pos[n]), end)

    # ---- bank colouring
    # entities: port bits of Block ports are coloured within capacity; bits of
    # explicit-register ports and nodes written to explicit output registers
    # are fixed; tied output nodes follow their input bit.
    fixed = {}
    cap_of = {}          # input node -> capacity key (group)
    capacity = {}
    for group, lits in C.inputs:
        spec = in_ports[group]
        if isinstance(spec, Block):
            capacity[group] = spec.capacity()
            for l in lits:
                cap_of[l >> 1] = group
        else:
            for l, r in zip(lits, spec):
                fixed[l >> 1] = bank(r)
    tie_of = {}          # node -> input node it must share a bank with
    for n, (group, b) in out_direct.items():
        spec = out_ports[group]
        if isinstance(spec, tuple):
            tied_group = spec[1]
            tie_of[n] = groups_in[tied_group][b] >> 1
        else:
            fixed[n] = bank(spec[b])
    nbr = defaultdict(set)
    for n in nodes:
        fan = C.fanins[n]
        for i in range(len(fan)):
            for j in range(i + 1, len(fan)):
                nbr[fan[i]].add(fan[j])
                nbr[fan[j]].add(fan[i])
    # a tied pair is coloured as one entity: merge neighbourhoods
    partner = {}
    for n, m in tie_of.items():
        partner[n] = m
        partner[m] = n
    color = dict(fixed)
    todo = set(n for n in list(nodes) + list(cap_of) if n not in color)
    load = [0] * NBANK

    def neighbours(n):
        s = set(nbr[n])
        if n in partner:
            s |= nbr[partner[n]]
        return s

    while todo:
        def key(n):
            cs = {color[m] for m in neighbours(n) if m in color}
            return (len(cs), len(neighbours(n)), n in cap_of or partner.get(n) in cap_of)
        n = max(todo, key=key)
        grp = cap_of.get(n) or cap_of.get(partner.get(n))
        cost = [0] * NBANK
        for m in neighbours(n):
            if m in color:
                cost[color[m]] += 1
        allowed = [b for b in range(NBANK) if grp is None or capacity[grp][b] > 0]
        if not allowed:
            raise AllocError(f"no bank capacity left for port {grp}")
        best = min(allowed, key=lambda b: (cost[b], load[b]))
        color[n] = best
        load[best] += 1
        if grp is not None:
            capacity[grp][best] -= 1
        todo.discard(n)
        if n in partner:
            color[partner[n]] = best
            todo.discard(partner[n])

    # ---- local search: move a value (with its tied partner) to another bank
    # when that lowers the number of instructions with a shared source bank
    movable = set(n for n in color if n not in fixed and n not in tie_of)
    users = defaultdict(list)
    for n in nodes:
        for f in C.fanins[n]:
            users[f].append(n)

    def bad(n):
        fan = C.fanins[n]
        return len(set(color[f] for f in fan)) < len(fan)

    for _ in range(8):
        improved = False
        for n in nodes:
            if not bad(n):
                continue
            for f in C.fanins[n]:
                if f not in movable:
                    continue
                grp = cap_of.get(f) or cap_of.get(partner.get(f))
                touched = set(users[f]) | (set(users[partner[f]]) if f in partner else set())
                before = sum(bad(u) for u in touched)
                old_c = color[f]
                for c in range(NBANK):
                    if c == old_c or (grp is not None and capacity[grp][c] == 0):
                        continue
                    color[f] = c
                    if f in partner:
                        color[partner[f]] = c
                    after = sum(bad(u) for u in touched)
                    if after < before:
                        if grp is not None:
                            capacity[grp][c] -= 1
                            capacity[grp][old_c] += 1
                        improved = True
                        break
                    color[f] = old_c
                    if f in partner:
                        color[partner[f]] = old_c
                if not bad(n):
                    break
        if not improved:
            break

    # ---- annealing: random single moves (a value with its tied partner),
    # accepted when they do not add conflicts or, with falling probability,
    # when they do; the best colouring seen is kept (fixed seed: the result
    # is reproducible)
    # A move recolours one value; within a port whose block is full it swaps
    # the banks of two of the port's bits instead.
    rng = np.random.default_rng(12345)
    mov = sorted(movable)
    members = defaultdict(list)
    for n in mov:
        g = cap_of.get(n) or cap_of.get(partner.get(n))
        if g is not None:
            members[g].append(n)

    def with_partner(n):
        return [n, partner[n]] if n in partner else [n]

    def set_color(ns, c):
        for m in ns:
            color[m] = c

    cur = sum(bad(u) for u in nodes)
    best_c, best_color = cur, dict(color)
    steps = 60 * len(mov) if cur else 0
    for step in range(steps):
        if best_c == 0:
            break
        temp = 0.6 * (1.0 - step / steps) + 0.02
        f = mov[int(rng.integers(len(mov)))]
        grp = cap_of.get(f) or cap_of.get(partner.get(f))
        old_c = color[f]
        if grp is not None and capacity[grp][old_c] == 0 and rng.random() < 0.5:
            g2 = members[grp][int(rng.integers(len(members[grp])))]
            c = color[g2]
            if c == old_c:
                continue
            moved = [(with_partner(f), old_c, c), (with_partner(g2), c, old_c)]
        else:
            c = int(rng.integers(NBANK))
            if c == old_c or (grp is not None and capacity[grp][c] == 0):
                continue
            moved = [(with_partner(f), old_c, c)]
        touched = set()
        for ns, _, _ in moved:
            for m in ns:
                touched |= set(users[m])
        before = sum(bad(u) for u in touched)
        for ns, _, new in moved:
            set_color(ns, new)
        delta = sum(bad(u) for u in touched) - before
        if delta <= 0 or rng.random() < np.exp(-delta / temp):
            cur += delta
            if grp is not None and len(moved) == 1:
                capacity[grp][c] -= 1
                capacity[grp][old_c] += 1
            if cur < best_c:
                best_c, best_color = cur, dict(color)
        else:
            for ns, old, _ in moved:
                set_color(ns, old)
    color = best_color

    # ---- place port bits
    pin, pout = {}, {}
    reg = {}
    for group, lits in C.inputs:
        spec = in_ports[group]
        if isinstance(spec, Block):
            avail = list(spec.regs)
            regs = []
            for l in lits:
                r = next(r for r in avail if bank(r) == color[l >> 1])
                avail.remove(r)
                regs.append(r)
        else:
            regs = list(spec)
        pin[group] = regs
        for l, r in zip(lits, regs):
            reg[l >> 1] = r
    out_reg = {}
    for group, lits in C.outputs:
        spec = out_ports[group]
        if spec == "pool":
            continue
        if isinstance(spec, tuple):
            blk, tied = spec
            in_blk = in_ports[tied]
            idx = [in_blk.regs.index(r) for r in pin[tied]]
            out_reg[group] = [blk.regs[i] for i in idx]
        else:
            out_reg[group] = list(spec)
        pout[group] = out_reg[group]
    placement = {"in": pin, "out": pout}
    in_set = set(r for regs in pin.values() for r in regs)
    out_set = set(r for regs in pout.values() for r in regs)
    if (in_set | out_set) & set(pool):
        raise AllocError("temporary pool overlaps port registers")
    # outputs are written while inputs may still be live: keep them disjoint
    if in_set & out_set:
        raise AllocError("output registers overlap input registers")

    # ---- linear scan
    free = {b: sorted(r for r in pool if bank(r) == b) for b in range(NBANK)}
    pool_set = set(pool)
    lines = []
    conflicts = 0
    off_bank = 0

    def take(b):
        nonlocal off_bank
        if free[b]:
            return free[b].pop(0)
        for alt in sorted(range(NBANK), key=lambda x: -len(free[x])):
            if free[alt]:
                off_bank += 1
                return free[alt].pop(0)
        raise AllocError("register pool exhausted")

    def release(v, i):
        if last.get(v, -1) == i and reg.get(v) in pool_set:
            r = reg[v]
            free[bank(r)].append(r)
            free[bank(r)].sort()

    for i, n in enumerate(nodes):
        fan = C.fanins[n]
        k = len(fan)
        tt = C.tts[n]
        for j, f in enumerate(fan):
            if f in flipped:
                tt = tt_flip(tt, k, j)
        if n in flipped:
            tt = ~tt & ((1 << (1 << k)) - 1)
        srcs = [f"v{reg[f]}" for f in fan]
        if len(set(bank(reg[f]) for f in fan)) < k:
            conflicts += 1
        for f in fan:
            release(f, i)
        if n in out_direct:
            g, b = out_direct[n]
            d = out_reg[g][b]
        else:
            d = take(color[n])
        reg[n] = d
        if k == 3:
            imm = tt
            ops = f"{srcs[2]}, {srcs[1]}, {srcs[0]}"
        elif k == 2:
            # f(x0, x1) as bitop3 of (S0, S1, S2) = (x1, x0, 0)
            imm = 0
            for s0 in range(2):
                for s1 in range(2):
                    if (tt >> (s1 | (s0 << 1))) & 1:
                        imm |= 1 << (s0 * 4 + s1 * 2)
            ops = f"{srcs[1]}, {srcs[0]}, 0"
        else:
            raise AllocError(f"node of arity {k}")
        lines.append(f"v_bitop3_b32 v{d}, {ops} bitop3:0x{imm:02x}")
    for g, lits in C.outputs:
        if out_ports[g] == "pool":
            pout[g] = [reg.get(l >> 1) for l in lits]
    for g, b, kind, src, inv in copies:
        if out_ports[g] == "pool":
            d = take(0)
            pout[g][b] = d
        else:
            d = out_reg[g][b]
        if kind == "const":
            lines.append(f"v_mov_b32 v{d}, {'-1' if src else '0'}")
        elif inv:
            lines.append(f"v_not_b32 v{d}, v{reg[src]}")
        else:
            lines.append(f"v_mov_b32 v{d}, v{reg[src]}")
    temps = sorted((set(reg.values()) | set(r for regs in pout.values() for r in regs))
                   & pool_set)
    stats = {"instructions": len(lines), "conflicts": conflicts, "off_bank": off_bank,
             "copies": sum(1 for c in copies if c[2] == "copy"), "temps": temps}
    return lines, placement, stats


# -- CPU interpreter of the emitted subset ---------------------------------------

def _bitop3(a, b, c, imm):
    out = np.zeros_like(a)
    for idx in range(8):
        if (imm >> idx) & 1:
            s0 = a if idx & 4 else ~a
            s1 = b if idx & 2 else ~b
            s2 = c if idx & 1 else ~c
            out |= s0 & s1 & s2
    return out


def _value(tok, regs, like):
    tok = tok.strip()
    if tok.startswith("v"):
        return regs[int(tok[1:])]
    v = int(tok, 0)
    return np.full_like(like, np.uint64(0xFFFFFFFFFFFFFFFF) if v == -1 else np.uint64(v))


def interpret(lines, regs):
    """Run instruction lines on a register file {reg: uint64 word array}
    (64 lanes per word here; every instruction is bitwise)."""
    like = next(iter(regs.values()))
    for ln in lines:
        op, rest = ln.split(None, 1)
        if op == "v_bitop3_b32":
            body, imm = rest.split(" bitop3:")
            d, a, b, c = [t.strip() for t in body.split(",")]
            regs[int(d[1:])] = _bitop3(_value(a, regs, like), _value(b, regs, like),
                                       _value(c, regs, like), int(imm, 16))
        elif op == "v_not_b32":
            d, a = [t.strip() for t in rest.split(",")]
            regs[int(d[1:])] = ~_value(a, regs, like)
        elif op == "v_mov_b32":
            d, a = [t.strip() for t in rest.split(",")]
            regs[int(d[1:])] = _value(a, regs, like).copy()
        else:
            raise ValueError(f"interpreter does not know {op}")
    return regs
