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
* resynthesis of small windows: a node whose function over a cut of four or
  five signals can be written as g(h(S), T) -- two LUTs, h over at most three
  of the signals and g over h and the other (at most two) -- while the part
  of its cone that nothing else uses holds more than two LUTs, gets that
  decomposition;
* substitution under don't-cares (``dont_care_substitute``): a node becomes a
  constant or an earlier signal wherever the two differ only on input
  patterns at which no output bit that matters can see the difference. Every
  input pattern is simulated, so the result is exact; it applies to circuits
  of at most 24 input bits;
* resubstitution under the same don't-cares (``resubstitute``): a node whose
  value, wherever an output bit that matters can see it, is a function of
  three earlier signals outside its fan-out-free cone becomes one LUT over
  them, and the cone's other LUTs go. Also exact, also up to 24 input bits.
"""
import itertools

import numpy as np

from . import sim
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


def _cofactor2(tt, k, i, vi, j, vj):
    """tt (k inputs) with inputs i < j fixed; the result is over the rest, in order."""
    return tt_cofactor(tt_cofactor(tt, k, j, vj), k - 1, i, vi)


def decompose2(tt, k):
    """f = g(h(S), T) for a k-input function (k = 4 or 5) whose inputs are all
    essential: T two inputs, S the other inputs, for k = 4 possibly with one
    input of T added. Returns (S, h_tt, T, g_tt), S and T as input indices
    (g's inputs are h, T[0], T[1]), or None."""
    for T in itertools.combinations(range(k), 2):
        R = [v for v in range(k) if v not in T]
        m = len(R)
        full = tt_mask(m)
        cof = [_cofactor2(tt, k, T[0], a & 1, T[1], a >> 1) for a in range(4)]
        # the non-constant cofactors, grouped by the value of the input of T
        # that h may also read (None: h reads R only)
        for shared in [None] + ([0, 1] if k == 4 else []):
            hs, kinds, ok = {}, [], True
            for a in range(4):
                c = cof[a]
                if c in (0, full):
                    kinds.append(c & 1)
                    continue
                key = None if shared is None else (a >> shared) & 1
                h = hs.setdefault(key, c)
                if c == h:
                    kinds.append("h")
                elif c == ~h & full:
                    kinds.append("~h")
                else:
                    ok = False
                    break
            if not ok or not hs:
                continue
            if shared is None:
                S, h_tt = R, next(iter(hs.values()))
            else:
                t = T[shared]
                S = sorted(R + [t])
                h_tt = 0
                for idx in range(8):
                    bits = {S[i]: (idx >> i) & 1 for i in range(3)}
                    r_idx = sum(bits[r] << i for i, r in enumerate(R))
                    h = hs.get(bits[t], 0)
                    h_tt |= ((h >> r_idx) & 1) << idx
            g_tt = 0
            for a in range(4):
                for hv in (0, 1):
                    kind = kinds[a]
                    out = hv if kind == "h" else (1 - hv if kind == "~h" else kind)
                    g_tt |= out << (hv | (a << 1))
            return list(S), h_tt, list(T), g_tt
    return None


def _mffc_size(C, n, leaves, fanout):
    """LUTs of n's cone above `leaves` that no node outside the cone uses."""
    refs = {}
    stop = set(leaves)
    count, stack = 0, [n]
    while stack:
        m = stack.pop()
        count += 1
        for f in C.fanins[m]:
            if f in stop or C.is_input[f] or f == 0:
                continue
            refs[f] = refs.get(f, 0) + 1
            if refs[f] == fanout[f]:
                stack.append(f)
    return count


def resynthesize(C: Circuit, max_steps=10000):
    """Apply the best two-LUT window decomposition (see decompose2) while
    one saves a LUT."""
    memo = {}
    for _ in range(max_steps):
        cuts = enumerate_cuts(C, k=5, limit=40)
        N = len(C.fanins)
        fanout = [0] * N
        for m in range(1, N):
            for f in C.fanins[m]:
                fanout[f] += 1
        for _, lits in C.outputs:
            for l in lits:
                fanout[l >> 1] += 1
        cands = []
        for n in range(1, N):
            if C.is_input[n]:
                continue
            for leaves, tt in cuts[n][:-1]:
                if len(leaves) < 4:
                    continue
                key = (tt, len(leaves))
                if key not in memo:
                    memo[key] = decompose2(tt, len(leaves))
                d = memo[key]
                if d is None:
                    continue
                gain = _mffc_size(C, n, leaves, fanout) - 2
                if gain > 0:
                    cands.append((gain, n, leaves, d))
        applied = False
        for gain, n, leaves, (S, h_tt, T, g_tt) in sorted(cands, key=lambda c: -c[0]):
            D = Circuit(C.name)
            m = {0: 0}
            for group, lits in C.inputs:
                for l, nl in zip(lits, D.input(group, len(lits))):
                    m[l >> 1] = nl
            for v in range(1, N):
                if C.is_input[v]:
                    continue
                if v == n:
                    h = D.lut(h_tt, [m[leaves[i]] for i in S])
                    m[v] = D.lut(g_tt, [h] + [m[leaves[i]] for i in T])
                else:
                    m[v] = D.lut(C.tts[v], [m[f] for f in C.fanins[v]])
            for group, lits in C.outputs:
                D.output(group, [m[l >> 1] ^ (l & 1) for l in lits])
            D = sweep(D)
            if D.n_nodes() < C.n_nodes():
                C, applied = D, True
                break
        if not applied:
            return C
    return C


def optimize(C: Circuit, max_iter=8, verbose=False):
    C = sweep(C)
    best = None
    for it in range(max_iter):
        C = functional_reduce(C)
        C = lut_map(C)
        C = resynthesize(C)
        n = C.n_nodes()
        if verbose:
            print(f"  iter {it}: {n} LUTs")
        if best is not None and n >= best.n_nodes():
            break
        best = C
    return best


def _node_values(C, planes):
    """Value of every node (uint64 word arrays) for input planes in port order."""
    v = {0: np.zeros_like(planes[0])}
    k = 0
    for _, lits in C.inputs:
        for l in lits:
            v[l >> 1] = planes[k]
            k += 1
    for n in range(1, len(C.fanins)):
        if not C.is_input[n]:
            fan = C.fanins[n]
            v[n] = sim._lut(C.tts[n], len(fan), [v[f] for f in fan])
    return v


def _out_values(C, v):
    return [~v[l >> 1] if l & 1 else v[l >> 1] for _, lits in C.outputs for l in lits]


def _visible(C, v, n, new, care, outs, fanout):
    """Patterns at which replacing node n's value by `new` changes a cared-for
    output bit (the transitive fan-out of n re-evaluated)."""
    w = {n: new}
    stack, seen = [n], {n}
    order = []
    while stack:
        m = stack.pop()
        for u in fanout[m]:
            if u not in seen:
                seen.add(u)
                order.append(u)
                stack.append(u)
    for u in sorted(order):
        fan = C.fanins[u]
        w[u] = sim._lut(C.tts[u], len(fan), [w.get(f, v[f]) for f in fan])
    diff = np.zeros_like(new)
    i = 0
    for _, lits in C.outputs:
        for l in lits:
            m = l >> 1
            if m in w:
                nv = ~w[m] if l & 1 else w[m]
                diff |= (nv ^ outs[i]) & care[i]
            i += 1
    return diff


def dont_care_substitute(C: Circuit, care_fn, max_inputs=24, samples=1 << 15, seed=1):
    """Replace nodes by a constant or by an earlier signal (either polarity)
    where no cared-for output can tell the difference.

    care_fn(outputs) -> one mask per output bit (word arrays like the
    outputs): the patterns at which that bit matters; it is evaluated on the
    circuit as given, whose outputs the masks then describe. Candidates are
    screened on random patterns and every substitution is checked on all
    2^inputs patterns before it is kept."""
    nin = sum(len(l) for _, l in C.inputs)
    if nin > max_inputs or nin < 6:
        return C
    full = sim.exhaustive_planes(nin)
    g = np.random.default_rng(seed)

    def sample(count):
        idx = g.integers(0, 1 << nin, count)
        planes = []
        for b in range(nin):
            bits = ((idx >> b) & 1).astype(np.uint8)
            planes.append(np.packbits(bits.reshape(-1, 64), axis=1, bitorder="little")
                          .view(np.uint64).reshape(-1))
        return planes

    # two random samples screen candidates before the exhaustive check
    samp, mid = sample(samples), sample(samples * 16)
    care_full = care_fn(_out_values(C, _node_values(C, full)))
    care_samp = care_fn(_out_values(C, _node_values(C, samp)))
    care_mid = care_fn(_out_values(C, _node_values(C, mid)))
    changed = True
    while changed:
        changed = False
        N = len(C.fanins)
        fanout = {m: [] for m in range(N)}
        for m in range(1, N):
            for f in C.fanins[m]:
                fanout[f].append(m)
        vs = _node_values(C, samp)
        outs_s = _out_values(C, vs)
        vm = outs_m = vf = outs_f = None
        # screen every node: the sample patterns where its value matters
        for n in range(N - 1, 0, -1):
            if C.is_input[n]:
                continue
            cs = _visible(C, vs, n, ~vs[n], care_samp, outs_s, fanout)
            t = vs[n]
            cands = []
            if not (t & cs).any():
                cands.append(0)                      # constant 0
            if not (~t & cs).any():
                cands.append(1)                      # constant 1
            for m in range(1, n):
                if not ((vs[m] ^ t) & cs).any():
                    cands.append(2 * m)
                elif not ((~vs[m] ^ t) & cs).any():
                    cands.append(2 * m + 1)
            if not cands:
                continue
            if vm is None:
                vm = _node_values(C, mid)
                outs_m = _out_values(C, vm)

            def survives(vals, care, outs, lit):
                base = vals[lit >> 1] if lit >> 1 else np.zeros_like(vals[n])
                new = ~base if lit & 1 else base
                return not _visible(C, vals, n, new, care, outs, fanout).any()

            cands = [lit for lit in cands if survives(vm, care_mid, outs_m, lit)]
            if cands and vf is None:
                vf = _node_values(C, full)
                outs_f = _out_values(C, vf)
            for lit in cands:
                if survives(vf, care_full, outs_f, lit):
                    D = rebuild(C, subst={n: lit})
                    if D.n_nodes() < C.n_nodes():
                        C, changed = D, True
                        break
            if changed:
                break
    return C


def noncanonical_care(wE, wF):
    """Output care masks of an operator whose result may be non-canonical:
    E and F matter only for a normal result, the sign unless it is NaN."""
    def care(outs):
        x0, x1 = outs[wE + wF + 1], outs[wE + wF + 2]
        normal, notnan = x0 & ~x1, ~(x0 & x1)
        every = np.full_like(x0, np.uint64(0xFFFFFFFFFFFFFFFF))
        return [normal] * (wE + wF) + [notnan, every, every]
    return care


def _fanout_lists(C):
    N = len(C.fanins)
    lists, counts = {m: [] for m in range(N)}, [0] * N
    for m in range(1, N):
        for f in C.fanins[m]:
            lists[f].append(m)
            counts[f] += 1
    for _, lits in C.outputs:
        for l in lits:
            counts[l >> 1] += 1
    return lists, counts


def _cone(C, n, counts):
    """The LUTs of n's maximum fan-out-free cone (n included)."""
    refs, cone, stack = {}, {n}, [n]
    while stack:
        m = stack.pop()
        for f in C.fanins[m]:
            if f == 0 or C.is_input[f]:
                continue
            refs[f] = refs.get(f, 0) + 1
            if refs[f] == counts[f]:
                cone.add(f)
                stack.append(f)
    return cone


def _function_of(t, care, xs):
    """Truth table over xs (at most three word arrays) that t follows on the
    patterns in care, or None; input combinations care never meets are 0."""
    tt = 0
    for idx in range(1 << len(xs)):
        m = care.copy()
        for i, x in enumerate(xs):
            m &= x if (idx >> i) & 1 else ~x
        if not m.any():
            continue
        one, zero = (m & t).any(), (m & ~t).any()
        if one and zero:
            return None
        if one:
            tt |= 1 << idx
    return tt


def _divisor_triples(t, care, V, names):
    """Triples of rows of V (in row order) that t is a function of on care."""
    D = V.shape[0]
    nt, nV = ~t, ~V
    out = []
    for i in range(D):
        for j in range(i + 1, D):
            ok = np.ones(D, bool)
            ok[:j + 1] = False
            for a in (V[i], nV[i]):
                for b in (V[j], nV[j]):
                    m = care & a & b
                    if not m.any():
                        continue
                    for c in (V, nV):
                        M = m & c
                        ok &= ~((M & t).any(axis=1) & (M & nt).any(axis=1))
            out.extend((names[i], names[j], names[int(k)]) for k in np.nonzero(ok)[0])
    return out


def resubstitute(C: Circuit, care_fn, max_inputs=24, max_divisors=160, seed=1):
    """One-LUT resubstitution under output don't-cares (care_fn as for
    dont_care_substitute). Largest cones first; the candidates come from 512
    random patterns, are screened on 2^15 more and checked on all 2^inputs
    patterns before the circuit is rebuilt; every accepted step removes at
    least one LUT. Divisors are the latest max_divisors earlier signals."""
    nin = sum(len(l) for _, l in C.inputs)
    if nin > max_inputs or nin < 6:
        return C
    g = np.random.default_rng(seed)

    def sample(count):
        idx = g.integers(0, 1 << nin, count)
        planes = []
        for b in range(nin):
            bits = ((idx >> b) & 1).astype(np.uint8)
            planes.append(np.packbits(bits.reshape(-1, 64), axis=1, bitorder="little")
                          .view(np.uint64).reshape(-1))
        return planes

    samp, mid, full = sample(512), sample(1 << 15), sim.exhaustive_planes(nin)
    care = [care_fn(_out_values(C, _node_values(C, p))) for p in (samp, mid, full)]
    changed = True
    while changed:
        changed = False
        N = len(C.fanins)
        fo, counts = _fanout_lists(C)
        vals = [_node_values(C, samp), None, None]
        outs = [_out_values(C, vals[0]), None, None]
        order = []
        for n in range(1, N):
            if not C.is_input[n]:
                cone = _cone(C, n, counts)
                if len(cone) >= 2:
                    order.append((len(cone), n, cone))
        order.sort(key=lambda c: (-c[0], c[1]))
        for _, n, cone in order:
            seen = _visible(C, vals[0], n, ~vals[0][n], care[0], outs[0], fo)
            if not seen.any():
                continue
            divs = [d for d in range(1, n) if d not in cone][-max_divisors:]
            cands = _divisor_triples(vals[0][n], seen, np.stack([vals[0][d] for d in divs]), divs)
            for level in (1, 2):
                if not cands:
                    break
                if vals[level] is None:
                    vals[level] = _node_values(C, (mid, full)[level - 1])
                    outs[level] = _out_values(C, vals[level])
                v = vals[level]
                seen = _visible(C, v, n, ~v[n], care[level], outs[level], fo)
                tts = [_function_of(v[n], seen, [v[d] for d in c]) for c in cands]
                cands = [c for c, tt in zip(cands, tts) if tt is not None]
                tts = [tt for tt in tts if tt is not None]
            for c, tt in zip(cands, tts if cands else []):
                D = Circuit(C.name)
                m = {0: 0}
                for group, lits in C.inputs:
                    for l, nl in zip(lits, D.input(group, len(lits))):
                        m[l >> 1] = nl
                for u in range(1, N):
                    if C.is_input[u]:
                        continue
                    if u == n:
                        m[u] = D.lut(tt, [m[d] for d in c])
                    else:
                        m[u] = D.lut(C.tts[u], [m[f] for f in C.fanins[u]])
                for group, lits in C.outputs:
                    D.output(group, [m[l >> 1] ^ (l & 1) for l in lits])
                D = sweep(D)
                if D.n_nodes() < C.n_nodes():
                    C, changed = D, True
                    break
            if changed:
                break
    return C
