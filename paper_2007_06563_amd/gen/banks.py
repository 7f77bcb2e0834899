"""VGPR bank pass over the device assembly the compiler writes.

A VALU instruction whose sources include two different VGPRs of one bank
(register number mod 4) takes about twice the SIMD's time once two or more
waves share the SIMD (measured with the library's issue-rate probe: 4.46
against 2.13 clocks per instruction). The split kernel's netlists are
allocated bank-aware by the generator; the fused conv kernel's MAC netlist is
compiled C++, and the compiler's allocation leaves about two in five of its
instructions with a bank clash.

This pass re-assigns the registers of values that live inside one basic block
(netlist temporaries): per block, every value defined by a plain bitwise VALU
instruction and read only by such instructions, and not live out of the
block, may move to another register of a pool that is free over its live
range. The choice minimises the number of instructions whose sources share a
bank, greedily over the values in program order, repeated until no choice
improves. Nothing else changes: instruction order, mnemonics, every operand
other than a moved value's register, and the kernel's VGPR count (the pool
holds only registers the function already uses).

Safety:
- liveness comes from a data-flow analysis over the function's control flow
  graph (branches and fall-throughs), with every instruction's VGPR reads and
  writes; a function with an instruction whose VGPR effects are not modelled,
  or with indirect branches, is left unchanged;
- the pool holds only registers that, in the whole function, are read and
  written by plain VALU instructions alone (never a memory instruction's
  destination, data or address, whose asynchronous completion a static view
  would not see);
- a block that writes EXEC is left alone, so every instruction of a block
  that is changed runs under one lane mask: a renamed value's lanes are
  written and read under the same mask, and lanes outside it are left
  untouched in every register, as before;
- after renaming, each block is checked against the original: every source
  operand must read the value of the same defining instruction (or the same
  incoming register), and every register live out of the block must hold the
  value of the same instruction. A block that fails is left as it was.
"""
import re

_LABEL = re.compile(r"^([A-Za-z_.$][\w.$]*):")
_VREG = re.compile(r"^v(\d+)$")
_VRANGE = re.compile(r"^v\[(\d+):(\d+)\]$")
_ANYV = re.compile(r"\bv(\d+)\b|\bv\[(\d+):(\d+)\]")

# plain bitwise / move VALU forms: one VGPR destination, operands that are
# single registers or constants, no implicit VGPR effects
_SIMPLE = re.compile(
    r"^v_(bitop3_b32|bfe_i32|bfe_u32|and_b32|or_b32|xor_b32|xnor_b32|not_b32|mov_b32|"
    r"alignbit_b32|lshlrev_b32|lshrrev_b32|ashrrev_i32|or3_b32|and_or_b32|lshl_or_b32|"
    r"xad_u32|bfi_b32|perm_b32|cndmask_b32)(_e32|_e64)?$")
_LOADS = ("ds_read", "ds_load", "global_load", "buffer_load", "flat_load", "scratch_load",
          "ds_swizzle", "ds_bpermute", "ds_permute")
_STORES = ("ds_write", "ds_store", "global_store", "buffer_store", "flat_store",
           "scratch_store")
_ATOMICS = ("global_atomic", "buffer_atomic", "flat_atomic", "ds_add", "ds_sub", "ds_inc",
            "ds_dec", "ds_min", "ds_max", "ds_and", "ds_or", "ds_xor", "ds_cmpst", "ds_wrxchg",
            "ds_cmpxchg")
_NO_VDST = ("v_cmp", "v_readfirstlane", "v_readlane", "v_nop")
_USE_DEF = ("v_writelane", "v_mac_", "v_fmac_")


def _split_ops(text):
    """Operands of one instruction, split at top-level commas."""
    out, depth, cur = [], 0, []
    for ch in text:
        if ch in "[(":
            depth += 1
        elif ch in "])":
            depth -= 1
        if ch == "," and depth == 0:
            out.append("".join(cur).strip())
            cur = []
        else:
            cur.append(ch)
    if cur and "".join(cur).strip():
        out.append("".join(cur).strip())
    return out


def _regs(op):
    """VGPR numbers named by one operand."""
    out = []
    for m in _ANYV.finditer(op):
        if m.group(1) is not None:
            out.append(int(m.group(1)))
        else:
            out.extend(range(int(m.group(2)), int(m.group(3)) + 1))
    return out


class Inst:
    __slots__ = ("line", "mn", "ops", "defs", "uses", "simple", "dst_single", "src_pos",
                 "branch", "target", "ends")

    def __init__(self, line, mn, ops):
        self.line, self.mn, self.ops = line, mn, ops
        self.defs, self.uses = [], []
        self.simple = False
        self.dst_single = None  # the single VGPR a simple instruction writes
        self.src_pos = []       # (operand index, register) of a simple instruction's sources
        self.branch = mn.startswith(("s_branch", "s_cbranch"))
        self.target = None
        self.ends = mn in ("s_endpgm", "s_branch") or mn.startswith(("s_setpc", "s_swappc"))


class Unmodelled(Exception):
    pass


def _writes_exec(inst):
    mn, ops = inst.mn, inst.ops
    return ("saveexec" in mn or mn.startswith("v_cmpx") or
            (mn.startswith("s_") and ops and ops[0].split()[0] in ("exec", "exec_lo", "exec_hi")))


def _effects(inst):
    """Fills defs/uses (lists of VGPR numbers) from the mnemonic's class."""
    mn, ops = inst.mn, inst.ops
    if mn.startswith(("v_movrel", "s_set_gpr_idx", "v_swap")):
        raise Unmodelled(mn)  # register indexing: any VGPR may be touched
    if not any(_ANYV.search(o) for o in ops):
        return
    first_tok = lambda o: o.split()[0] if o else o
    if _SIMPLE.match(mn):
        m = _VREG.match(first_tok(ops[0]))
        toks = [first_tok(o) for o in ops[1:]]
        single = all(_VREG.match(t) or not _ANYV.search(o) for t, o in zip(toks, ops[1:]))
        if m and single and not any(" " in o and _ANYV.search(o.split(None, 1)[1]) for o in ops):
            inst.simple = True
            inst.dst_single = int(m.group(1))
            inst.defs = [inst.dst_single]
            for j, o in enumerate(ops[1:], start=1):
                mm = _VREG.match(first_tok(o))
                if mm:
                    inst.src_pos.append((j, int(mm.group(1))))
                    inst.uses.append(int(mm.group(1)))
            return
    if mn.startswith("v_"):
        if mn.startswith(_NO_VDST):
            inst.uses = [r for o in ops for r in _regs(o)]
            return
        d = _regs(ops[0])
        u = [r for o in ops[1:] for r in _regs(o)]
        if mn.startswith(_USE_DEF) or mn.endswith("_sdwa"):
            u += d
        inst.defs, inst.uses = d, u
        return
    if mn.startswith(_ATOMICS):
        allr = [r for o in ops for r in _regs(o)]
        inst.defs, inst.uses = allr, allr
        return
    if mn.startswith(_LOADS):
        d = _regs(ops[0])
        u = [r for o in ops[1:] for r in _regs(o)]
        if "d16" in mn:
            u += d
        inst.defs, inst.uses = d, u
        return
    if mn.startswith(_STORES):
        inst.uses = [r for o in ops for r in _regs(o)]
        return
    raise Unmodelled(mn)


def _parse_function(lines, lo, hi):
    """Instructions and labels of lines[lo:hi]: (insts, label -> index of the
    first instruction after it)."""
    insts, labels = [], {}
    for i in range(lo, hi):
        s = lines[i].split(";", 1)[0].strip()
        if not s:
            continue
        m = _LABEL.match(s)
        if m:
            labels[m.group(1)] = len(insts)
            if s[m.end():].strip():
                raise Unmodelled("label with code")
            continue
        if s.startswith("."):
            continue
        parts = s.split(None, 1)
        inst = Inst(i, parts[0], _split_ops(parts[1]) if len(parts) > 1 else [])
        _effects(inst)
        if inst.branch:
            inst.target = inst.ops[0] if inst.ops else None
        insts.append(inst)
    return insts, labels


def _blocks(insts, labels):
    """Basic blocks as (start, end) index ranges and their successors."""
    starts = {0} | set(labels.values())
    for k, ins in enumerate(insts):
        if ins.branch or ins.ends:
            starts.add(k + 1)
    starts = sorted(s for s in starts if s < len(insts))
    blocks = []
    for j, s in enumerate(starts):
        e = starts[j + 1] if j + 1 < len(starts) else len(insts)
        blocks.append((s, e))
    index_of = {s: j for j, (s, _) in enumerate(blocks)}
    succ = []
    for j, (s, e) in enumerate(blocks):
        last = insts[e - 1]
        out = []
        if last.mn.startswith(("s_setpc", "s_swappc")):
            raise Unmodelled("indirect branch")
        if last.branch:
            if last.target not in labels or labels[last.target] not in index_of:
                raise Unmodelled(f"branch target {last.target}")
            out.append(index_of[labels[last.target]])
        if not (last.mn in ("s_endpgm", "s_branch")) and j + 1 < len(blocks):
            out.append(j + 1)
        succ.append(out)
    return blocks, succ


def _liveness(insts, blocks, succ):
    use_b, def_b = [], []
    for s, e in blocks:
        u, d = set(), set()
        for ins in insts[s:e]:
            u |= set(ins.uses) - d
            d |= set(ins.defs)
        use_b.append(u)
        def_b.append(d)
    live_in = [set() for _ in blocks]
    live_out = [set() for _ in blocks]
    changed = True
    while changed:
        changed = False
        for j in reversed(range(len(blocks))):
            out = set()
            for t in succ[j]:
                out |= live_in[t]
            inn = use_b[j] | (out - def_b[j])
            if out != live_out[j] or inn != live_in[j]:
                live_out[j], live_in[j] = out, inn
                changed = True
    return live_in, live_out


def _reaching(seq, regs_of, live_out):
    """Per instruction of a block, the defining instruction (or 'in') of each
    source register read; and of each live-out register at the end."""
    last = {}
    reads = []
    for k, (defs, uses) in enumerate(seq):
        reads.append(tuple(last.get(r, ("in", regs_of(r))) for r in uses))
        for r in defs:
            last[r] = k
    outs = {}
    for r in live_out:
        outs[r] = last.get(r, ("in", r))
    return reads, outs


def _conflicting(regs):
    banks = [r & 3 for r in set(regs)]
    return len(banks) != len(set(banks))


def _rename_block(insts, s, e, live_in, live_out, pool, max_passes=6):
    """Returns {(inst index, operand index): new register} for one block, or
    {} if nothing improves or the check fails."""
    n = e - s
    B = insts[s:e]
    # values: (def position k, register, last use, use positions, renameable)
    last_def = {}
    for k, ins in enumerate(B):
        for r in ins.defs:
            last_def[r] = k
    values = []
    open_val = {}  # register -> value currently held
    # incoming values
    for r in pool:
        if r in live_in:
            v = {"k": -1, "r": r, "u": -1, "uses": [], "ren": False}
            open_val[r] = v
            values.append(v)
    for k, ins in enumerate(B):
        for r in set(ins.uses):
            v = open_val.get(r)
            if v is not None:
                v["uses"].append(k)
                v["u"] = k
        for r in ins.defs:
            if r not in pool:
                open_val.pop(r, None)
                continue
            v = {"k": k, "r": r, "u": k, "uses": [], "ren": ins.simple and r == ins.dst_single}
            open_val[r] = v
            values.append(v)
    for r, v in open_val.items():
        if r in live_out:
            v["u"] = n  # live past the block end
            v["ren"] = False
    for v in values:
        if v["ren"] and not all(B[u].simple for u in v["uses"]):
            v["ren"] = False
    # registers of the pool untouched here but live through the block
    touched = {v["r"] for v in values}
    for r in pool:
        if r not in touched and r in live_out:
            values.append({"k": -1, "r": r, "u": n, "uses": [], "ren": False})
    ren = [v for v in values if v["ren"]]
    if not ren:
        return {}
    occ = {r: [] for r in pool}
    for v in values:
        occ[v["r"]].append(v)
    cur = {id(v): v["r"] for v in values}
    # which value each (position, register) source reads
    reader = {}
    for v in values:
        for u in v["uses"]:
            reader[(u, v["r"])] = v

    def src_regs(k, skip=None):
        out = []
        for r in set(B[k].uses):
            w = reader.get((k, r))
            if w is skip and w is not None:
                continue
            out.append(cur[id(w)] if w is not None else r)
        return out

    def cost(v, p):
        c = 0
        for u in v["uses"]:
            others = src_regs(u, skip=v)
            if any((q & 3) == (p & 3) and q != p for q in others):
                c += 1
        return c

    def free(p, v):
        for w in occ[p]:
            if w is v:
                continue
            if w["k"] < v["u"] and v["k"] < w["u"]:
                return False
            if w["k"] == v["k"]:
                return False
        return True

    def total():
        return sum(1 for k in range(n) if B[k].mn.startswith("v_") and _conflicting(src_regs(k)))

    before = total()
    for _ in range(max_passes):
        improved = False
        for v in sorted(ren, key=lambda v: v["k"]):
            p0 = cur[id(v)]
            occ[p0].remove(v)
            best = (cost(v, p0), 0, p0)
            for p in pool:
                if p == p0 or not free(p, v):
                    continue
                c = (cost(v, p), 1, p)
                if c < best:
                    best = c
            cur[id(v)] = best[2]
            occ[best[2]].append(v)
            if best[2] != p0:
                improved = True
        if not improved:
            break
    after = total()
    if after >= before:
        return {}
    # the renamed block's register effects
    newreg = {}
    for v in values:
        if cur[id(v)] != v["r"]:
            newreg[(v["k"], "def")] = cur[id(v)]
            for u in v["uses"]:
                newreg[(u, v["r"])] = cur[id(v)]
    seq_old, seq_new = [], []
    for k, ins in enumerate(B):
        seq_old.append((ins.defs, ins.uses))
        d = [newreg.get((k, "def"), r) if (ins.simple and r == ins.dst_single) else r
             for r in ins.defs]
        u = [newreg.get((k, r), r) for r in ins.uses]
        seq_new.append((d, u))
    # check: same producers for every read and for every live-out register
    r_old, o_old = _reaching(seq_old, lambda r: r, live_out)
    # map incoming registers of the new sequence back to themselves
    r_new, o_new = _reaching(seq_new, lambda r: r, live_out)
    if r_old != r_new or o_old != o_new:
        return {}
    edits = {}
    for k, ins in enumerate(B):
        if (k, "def") in newreg and ins.simple:
            edits[(s + k, 0)] = newreg[(k, "def")]
        for j, r in ins.src_pos:
            if (k, r) in newreg:
                edits[(s + k, j)] = newreg[(k, r)]
    return edits, before, after


def rename_text(text, only=None, max_reg=None):
    """Returns (new_text, stats). Functions are the code sections whose name
    contains one of `only` (all code sections if None)."""
    lines = text.split("\n")
    stats = {"functions": 0, "skipped": 0, "blocks": 0, "conflicts_before": 0,
             "conflicts_after": 0}
    # function extents: a code section from its label to the next section
    spans, cur, start = [], None, None
    for i, raw in enumerate(lines):
        s = raw.strip()
        if s.startswith(".section") or s in (".text", ".data", ".bss"):
            if cur is not None:
                spans.append((cur, start, i))
            name = s.split(None, 1)[1].split(",", 1)[0].strip() if s.startswith(".section") else s
            cur, start = (name, i) if name.startswith(".text") else (None, None)
    if cur is not None:
        spans.append((cur, start, len(lines)))
    for name, lo, hi in spans:
        if only is not None and not any(k in name for k in only):
            continue
        try:
            insts, labels = _parse_function(lines, lo, hi)
            blocks, succ = _blocks(insts, labels)
        except Unmodelled:
            stats["skipped"] += 1
            continue
        if not insts:
            continue
        stats["functions"] += 1
        live_in, live_out = _liveness(insts, blocks, succ)
        used = set()
        pinned = set()
        for ins in insts:
            used |= set(ins.defs) | set(ins.uses)
            if not ins.simple:
                pinned |= set(ins.defs) | set(ins.uses)
        top = max(used) if used else -1
        if max_reg is not None:
            top = min(top, max_reg)
        pool = sorted(r for r in range(top + 1) if r not in pinned)
        pool_set = set(pool)
        for j, (s, e) in enumerate(blocks):
            # a block that changes EXEC part-way would mix lane sets: left alone
            if any(_writes_exec(ins) for ins in insts[s:e]):
                continue
            res = _rename_block(insts, s, e, live_in[j], live_out[j], pool_set)
            if not res:
                continue
            edits, before, after = res
            stats["blocks"] += 1
            stats["conflicts_before"] += before
            stats["conflicts_after"] += after
            by_inst = {}
            for (k, j2), p in edits.items():
                by_inst.setdefault(k, {})[j2] = p
            for k, ch in by_inst.items():
                ins = insts[k]
                ops = list(ins.ops)
                for j2, p in ch.items():
                    tok = ops[j2].split(None, 1)
                    tok[0] = f"v{p}"
                    ops[j2] = " ".join(tok)
                indent = lines[ins.line][:len(lines[ins.line]) - len(lines[ins.line].lstrip())]
                comment = ""
                if ";" in lines[ins.line]:
                    comment = " ;" + lines[ins.line].split(";", 1)[1]
                lines[ins.line] = f"{indent}{ins.mn} {', '.join(ops)}{comment}"
    return "\n".join(lines), stats


def count_conflicts(text, only=None):
    """Instructions of the selected code sections whose VGPR sources share a
    bank (a diagnostic for tests and the build log)."""
    lines = text.split("\n")
    n, cur = 0, None
    for raw in lines:
        s = raw.split(";", 1)[0].strip()
        if s.startswith(".section") or s in (".text", ".data", ".bss"):
            name = s.split(None, 1)[1].split(",", 1)[0].strip() if s.startswith(".section") else s
            cur = name if name.startswith(".text") and (
                only is None or any(k in name for k in only)) else None
            continue
        if cur is None or not s.startswith("v_"):
            continue
        parts = s.split(None, 1)
        if len(parts) < 2:
            continue
        ops = _split_ops(parts[1])
        srcs = []
        for o in ops[1:]:
            m = _VREG.match(o.split()[0]) if o else None
            if m:
                srcs.append(int(m.group(1)))
        n += _conflicting(srcs)
    return n
