"""Netlist optimisation and 3-input LUT mapping.

The paper minimises gate count with commercial synthesis against a cell
library of the target's bitwise instructions, then restructures with an AIG
optimiser (Sec. 3.3). Neither tool exists here, so this module does the same
job for a cell library in which *every* function of up to three inputs costs
one instruction (gfx950 ``v_bitop3_b32``):

* cut enumeration: for each node, the sets of at most K signals that
  determine it, with the node's truth table over each set;
* functional reduction: a node whose cut function is a constant, a single
  signal, or equal (up to complement) to an earlier node's function on the
  same cut is replaced by that signal;
* area-oriented cut mapping with exact-area recovery: choose one cut per
  mapped node so that the number of LUTs is smallest;
* resynthesis of small windows: a node whose function over up to five inputs
  admits a cheaper two- or three-LUT decomposition than its current cone gets
  that decomposition.
"""
import itertools

from .circuit import Circuit, normalize, tt_mask, tt_var, tt_depends, tt_cofactor

K = 3


def compose(tt, k, subs, m):
    """tt (k inputs) applied to the k functions subs (each over m inputs)."""
    out = 0
    full = tt_mask(m)
    for idx in range(1 << k):
        if not (tt >> idx) & 1:
            continue
        term = full
        for i in range(k):
            term &= subs[i] if (idx >> i) & 1 else (~subs[i] & full)
        out |= term
    return out


def expand(tt, leaves, union):
    """Function tt over `leaves` re-expressed over `union` (a superset)."""
    m = len(union)
    subs = [tt_var(m, union.index(l)) for l in leaves]
    return compose(tt, len(leaves), subs, m)


def reduce_cut(leaves, tt):
    leaves = list(leaves)
    i = 0
    while i < len(leaves):
        if not tt_depends(tt, len(leaves), i):
            tt = tt_cofactor(tt, len(leaves), i, 0)
            del leaves[i]
        else:
            i += 1
    return tuple(leaves), tt


def enumerate_cuts(C: Circuit, k=K, limit=24):
    """cuts[n] = list of (leaves, tt), smallest first; the trivial cut last."""
    cuts = [None] * len(C.fanins)
    for n in range(1, len(C.fanins)):
        if C.is_input[n]:
            cuts[n] = [((n,), 0b10)]
            continue
        fan = C.fanins[n]
        seen = {}
        for combo in itertools.product(*[cuts[f] for f in fan]):
            union = sorted(set().union(*[c[0] for c in combo]))
            if len(union) > k:
                continue
            subs = [expand(c[1], c[0], union) for c in combo]
            tt = compose(C.tts[n], len(fan), subs, len(union))
            leaves, tt = reduce_cut(union, tt)
            if leaves not in seen:
                seen[leaves] = tt
        # drop dominated cuts (a superset of another cut's leaves)
        keys = sorted(seen, key=len)
        kept = []
        for ls in keys:
            s = set(ls)
            if any(set(o) <= s for o in kept):
                continue
            kept.append(ls)
        kept = kept[:limit]
        cuts[n] = [(ls, seen[ls]) for ls in kept] + [((n,), 0b10)]
    return cuts


def rebuild(C: Circuit, subst=None, cover=None, name=None):
    """A new circuit from C: nodes in `subst` are replaced by another old
    literal; with `cover`, only covered nodes are built, from their cuts."""
    D = Circuit(name or C.name)
    m = {0: 0}
    for group, lits in C.inputs:
        new = D.input(group, len(lits))
        for l, nl in zip(lits, new):
            m[l >> 1] = nl

    def lit(l):
        return m[l >> 1] ^ (l & 1)

    if cover is None:
        for n in range(1, len(C.fanins)):
            if C.is_input[n]:
                continue
            if subst and n in subst:
                m[n] = lit(subst[n])
            else:
                m[n] = D.lut(C.tts[n], [lit(2 * f) for f in C.fanins[n]])
    else:
        for n in sorted(cover):
            leaves, tt = cover[n]
            m[n] = D.lut(tt, [lit(2 * l) for l in leaves])
    for group, lits in C.outputs:
        D.output(group, [lit(l) for l in lits])
    return sweep(D)


def sweep(C: Circuit):
    """Drop nodes no output depends on (renumbering in topological order)."""
    live = set()
    stack = [l >> 1 for _, ls in C.outputs for l in ls]
    while stack:
        n = stack.pop()
        if n in live:
            continue
        live.add(n)
        stack.extend(C.fanins[n])
    if all((n in live) or C.is_input[n] or n == 0 for n in range(len(C.fanins))):
        return C
    D = Circuit(C.name)
    m = {0: 0}
    for group, lits in C.inputs:
        new = D.input(group, len(lits))
        for l, nl in zip(lits, new):
            m[l >> 1] = nl
    for n in range(1, len(C.fanins)):
        if C.is_input[n] or n not in live:
            continue
        m[n] = D.lut(C.tts[n], [m[f] for f in C.fanins[n]])
    for group, lits in C.outputs:
        D.output(group, [m[l >> 1] ^ (l & 1) for l in lits])
    return D


def functional_reduce(C: Circuit):
    """Merge nodes that are constant, a copy of one signal, or equal up to
    complement to an earlier node, as seen on some common cut."""
    while True:
        cuts = enumerate_cuts(C)
        subst = {}
        index = {}
        for n in range(1, len(C.fanins)):
            if C.is_input[n]:
                continue
            rep = None
            for leaves, tt in cuts[n][:-1]:
                k = len(leaves)
                if k == 0:
                    rep = tt & 1
                    break
                if k == 1 and tt in (1, 2) and leaves[0] != n:
                    rep = 2 * leaves[0] + (tt == 1)
                    break
                full = tt_mask(k)
                for t, inv in ((tt, 0), (~tt & full, 1)):
                    other = index.get((leaves, t))
                    if other is not None and other != n:
                        rep = 2 * other + inv
                        break
                if rep is not None:
                    break
            if rep is not None:
                subst[n] = rep
                continue
            for leaves, tt in cuts[n][:-1]:
                index.setdefault((leaves, tt), n)
        if not subst:
            return C
        C = rebuild(C, subst=subst)


def lut_map(C: Circuit, rounds=3):
    """Area-oriented mapping into <=3-input LUTs; returns the mapped circuit."""
    cuts = enumerate_cuts(C)
    N = len(C.fanins)
    fanout = [0] * N
    for n in range(1, N):
        for f in C.fanins[n]:
            fanout[f] += 1
    for _, lits in C.outputs:
        for l in lits:
            fanout[l >> 1] += 1
    # area flow
    af = [0.0] * N
    best = [None] * N
    for n in range(1, N):
        if C.is_input[n]:
            continue
        bc, bv = None, None
        for c in cuts[n][:-1]:
            v = 1.0 + sum(af[l] / max(fanout[l], 1) for l in c[0])
            if bv is None or v < bv - 1e-9 or (abs(v - bv) < 1e-9 and len(c[0]) < len(bc[0])):
                bc, bv = c, v
        best[n], af[n] = bc, bv
    refs = [0] * N

    def ref(n):
        """Reference n; returns the number of LUTs newly needed."""
        if n == 0 or C.is_input[n]:
            return 0
        refs[n] += 1
        if refs[n] > 1:
            return 0
        return 1 + sum(ref(l) for l in best[n][0])

    def deref(n):
        if n == 0 or C.is_input[n]:
            return 0
        refs[n] -= 1
        if refs[n] > 0:
            return 0
        return 1 + sum(deref(l) for l in best[n][0])

    for _, lits in C.outputs:
        for l in lits:
            ref(l >> 1)
    for _ in range(rounds):
        for n in range(1, N):
            if C.is_input[n] or refs[n] == 0:
                continue
            # free n's current cone, then price every cut by the LUTs it adds
            for l in best[n][0]:
                deref(l)
            chosen, cost = None, None
            for c in cuts[n][:-1]:
                save = best[n]
                best[n] = c
                a = sum(ref(l) for l in c[0])
                for l in c[0]:
                    deref(l)
                best[n] = save
                if cost is None or a < cost:
                    chosen, cost = c, a
            best[n] = chosen
            for l in chosen[0]:
                ref(l)
    cover = {n: best[n] for n in range(1, N) if not C.is_input[n] and refs[n] > 0}
    return rebuild(C, cover=cover)


def optimize(C: Circuit, max_iter=8, verbose=False):
    C = sweep(C)
    best = None
    for it in range(max_iter):
        C = functional_reduce(C)
        C = lut_map(C)
        n = C.n_nodes()
        if verbose:
            print(f"  iter {it}: {n} LUTs")
        if best is not None and n >= best:
            break
        best = n
    return C
