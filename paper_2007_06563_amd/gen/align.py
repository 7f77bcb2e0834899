"""Instruction alignment pass over the device assembly the compiler writes.

On gfx950 a wave issues an 8-byte instruction (VOP3 such as v_bitop3_b32, DS,
global memory, SMEM) about one clock later when it starts at an address that
is 4 mod 8: a straight run of such instructions issues every ~5 clocks
instead of every 4, while the same run at 8-byte aligned addresses, or a run
of 4-byte instructions, issues every 4 (measured with the library's
issue-rate probe). The compiler does not track this, and a bitsliced netlist
that mixes 4-byte VOP2 gates (v_and_b32, v_xor_b32, ...) with 8-byte
v_bitop3_b32 ends up with most of its 8-byte instructions misaligned.

The pass walks each code section in address order and, wherever the next
8-byte instruction would start at 4 mod 8, re-encodes one 4-byte VALU
instruction of the 4-byte run in front of it in its 8-byte VOP3 form (the
same operation on the same operands: `v_xor_b32_e32` becomes
`v_xor_b32_e64`). Where the run holds no such instruction (only SALU or
waits), it inserts one `s_nop 0` at the head of the run. Instruction sizes
come from the assembler itself (`llvm-mc -show-encoding`), so nothing here
guesses an encoding. A section with program-counter arithmetic whose next
instruction could move is left alone.

The penalty is a single wave's: with several waves on a SIMD, the SIMD
issues another wave's instruction meanwhile and misalignment costs little,
while an inserted s_nop still takes an issue slot. The build therefore runs
the pass only on the kernels measured faster with it.
"""
import re
import subprocess

# 4-byte VALU forms whose 8-byte VOP3 form takes the same operand text; carry
# ops, exec-writing compares and the like are not touched
_E32 = re.compile(r"^v_[a-z0-9_]+_e32$")
_EXCLUDE = ("v_cmpx_", "v_add_co_", "v_addc_co_", "v_sub_co_", "v_subb_co_", "v_subrev_co_",
            "v_subbrev_co_", "v_div_", "v_swap_", "v_accvgpr", "v_dot", "v_fmac_", "v_mac_",
            "v_pk_", "v_madmk", "v_madak", "v_fmamk", "v_fmaak", "v_readfirstlane", "v_nop",
            "v_movrel", "v_permlane")
_PC_OPS = ("s_getpc_b64", "s_setpc_b64", "s_swappc_b64")
_LABEL = re.compile(r"^[A-Za-z_.$][\w.$]*:")


def promotable(mnemonic):
    return bool(_E32.match(mnemonic)) and not mnemonic.startswith(_EXCLUDE)


def _classify(lines):
    """Yields (index, kind, payload) for the lines that matter: ('section',
    name), ('align', log2), ('inst', mnemonic)."""
    in_meta = False  # the YAML metadata block is text, not code
    for i, raw in enumerate(lines):
        s = raw.split(";", 1)[0].strip()
        if in_meta:
            in_meta = s != ".end_amdgpu_metadata"
            continue
        if not s:
            continue
        if s == ".amdgpu_metadata":
            in_meta = True
            continue
        if s.startswith("."):
            tok = s.split(None, 1)
            d = tok[0]
            if d == ".section":
                yield i, "section", tok[1].split(",", 1)[0].strip()
            elif d in (".text", ".data", ".bss"):
                yield i, "section", d
            elif d == ".p2align":
                yield i, "align", int(tok[1].split(",", 1)[0])
            elif d in (".align", ".balign", ".byte", ".short", ".long", ".quad", ".zero",
                       ".fill", ".space", ".skip", ".word", ".4byte", ".8byte"):
                yield i, "data", d
            continue
        m = _LABEL.match(s)
        if m:
            if s[m.end():].strip():
                yield i, "data", "label with code"
            continue
        yield i, "inst", s.split(None, 1)[0]


def encoding_sizes(asm_path, llvm_mc, mcpu="gfx950"):
    """Byte size of every instruction of the file, in order, from the
    assembler's own encoding listing."""
    r = subprocess.run([llvm_mc, "-triple=amdgcn-amd-amdhsa", f"-mcpu={mcpu}", "-show-encoding",
                        asm_path, "-o", "-"], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"llvm-mc failed on {asm_path}:\n{r.stderr[-2000:]}")
    out = []
    for line in r.stdout.splitlines():
        k = line.find("; encoding: [")
        if k >= 0:
            # bytes, some of them fixups ("A") for a label operand
            body = line[k + len("; encoding: ["):line.index("]", k)]
            out.append((line[:k].split(None, 1)[0], len(body.split(","))))
    return out


def _same_op(s_mn, mc_mn):
    return mc_mn == s_mn or mc_mn.startswith(s_mn + "_e") or s_mn.startswith(mc_mn)


# An s_nop 0 takes an issue slot (about four clocks); a misaligned 8-byte
# instruction costs about one. A nop is inserted only in front of a stretch of
# at least this many 8-byte instructions that would otherwise stay misaligned.
kNopWorth = 4


def _misaligned_stretch(seq, j, size_of):
    """8-byte instructions from seq[j] on that stay misaligned when nothing is
    changed: up to the next 4-byte run that restores the parity by itself or
    holds a promotable instruction, or the next alignment directive."""
    count, n = 0, len(seq)
    while j < n:
        it = seq[j]
        if it[1] == "align":
            if it[2] >= 3:
                return count
            j += 1
            continue
        sz = size_of[it[0]]
        if sz % 8 == 0:
            count += 1
            j += 1
            continue
        k, odd, prom = j, 0, False
        while k < n and seq[k][1] == "inst" and size_of[seq[k][0]] % 8 == 4:
            odd ^= 1
            prom = prom or promotable(seq[k][2])
            k += 1
        if odd or prom:
            return count
        j = k
    return count


def align_text(text, sizes, only=None):
    """Returns (new_text, stats). `sizes` is encoding_sizes() of `text`.
    only: if given, only the code sections whose name contains one of these
    strings are changed."""
    lines = text.split("\n")
    items = list(_classify(lines))
    insts = [it for it in items if it[1] == "inst"]
    stats = {"promoted": 0, "nops": 0, "left": 0, "skipped_sections": 0}
    if len(insts) != len(sizes) or any(not _same_op(it[2], mc) for it, (mc, _) in
                                       zip(insts, sizes)):
        raise RuntimeError("instruction lines and assembler encodings do not line up "
                           f"({len(insts)} lines, {len(sizes)} encodings)")
    size_of = {}
    for it, (_, n) in zip(insts, sizes):
        size_of[it[0]] = n
    # group the items by section, in file order (a section may be entered
    # more than once; its address counter carries over)
    by_sec, order, cur = {}, [], None
    for it in items:
        if it[1] == "section":
            cur = it[2]
            if cur not in by_sec:
                by_sec[cur] = []
                order.append(cur)
            continue
        if cur is not None:
            by_sec[cur].append(it)
    promote, nop_before = set(), set()
    for sec in order:
        if not sec.startswith(".text") or (only is not None and not any(k in sec for k in only)):
            continue
        seq = by_sec[sec]
        if any(it[1] == "data" for it in seq) or any(
                it[1] == "inst" and it[2] in _PC_OPS and
                (k + 1 >= len(seq) or size_of.get(seq[k + 1][0], 4) % 8 == 4)
                for k, it in enumerate(seq)):
            # program-counter arithmetic whose next instruction could move
            stats["skipped_sections"] += 1
            continue
        a, n, i = 0, len(seq), 0
        while i < n:
            it = seq[i]
            if it[1] == "align":
                a = -(-a // (1 << it[2])) * (1 << it[2])
                i += 1
                continue
            sz = size_of[it[0]]
            if sz % 4:
                raise RuntimeError(f"instruction of {sz} bytes: {lines[it[0]].strip()}")
            if sz % 8 == 0:
                a += sz
                i += 1
                continue
            # a run of instructions that flip the address parity, up to the
            # next 8-byte instruction or alignment directive
            j, run = i, []
            while j < n and seq[j][1] == "inst" and size_of[seq[j][0]] % 8 == 4:
                run.append(seq[j])
                j += 1
            end = a + sum(size_of[r[0]] for r in run)
            if j < n and seq[j][1] == "inst" and end % 8 == 4:
                cand = [r for r in run if promotable(r[2])]
                if cand:
                    promote.add(cand[-1][0])
                    stats["promoted"] += 1
                    end += 4
                elif _misaligned_stretch(seq, j, size_of) >= kNopWorth:
                    nop_before.add(run[0][0])
                    stats["nops"] += 1
                    end += 4
                else:
                    stats["left"] += 1
            a = end
            i = j
    for idx in promote:
        mn = lines[idx].split(";", 1)[0].split()[0]
        lines[idx] = lines[idx].replace(mn, mn[:-4] + "_e64", 1)
    for idx in sorted(nop_before, reverse=True):
        lines.insert(idx, "\ts_nop 0")
    return "\n".join(lines), stats


def misaligned_8byte(sizes_with_align, text):
    """Counts 8-byte instructions at addresses 4 mod 8 in the code sections of
    `text` (sizes as from encoding_sizes(text))."""
    lines = text.split("\n")
    items = list(_classify(lines))
    insts = [it for it in items if it[1] == "inst"]
    size_of = {it[0]: n for it, (_, n) in zip(insts, sizes_with_align)}
    addr, cur, count, total = {}, None, 0, 0
    for it in items:
        if it[1] == "section":
            cur = it[2]
            addr.setdefault(cur, 0)
            continue
        if cur is None or not cur.startswith(".text"):
            continue
        if it[1] == "align":
            m = 1 << it[2]
            addr[cur] = -(-addr[cur] // m) * m
        elif it[1] == "inst":
            sz = size_of[it[0]]
            if sz == 8:
                total += 1
                count += addr[cur] % 8 != 0
            addr[cur] += sz
    return count, total
