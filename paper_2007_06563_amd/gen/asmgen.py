"""Inline-assembly device functions for the split convolution kernel.

The two wave roles of the split kernel run their netlists as inline assembly
with explicit registers chosen by gen.regalloc, so that no VALU instruction
reads two VGPRs of one bank (see gen/regalloc.py). The functions produced:

* ``accum_loop(acc, e0, e1, e2, fl, nb, cap, gave)``: the whole accumulator
  role. Batch b (K products) sits in slot b % kSlots of the LDS product ring;
  its entries are requested with 16-byte loads at immediate offsets from this
  lane's first entry, on the schedule split_functions is given, and K copies
  of the adder netlist add them into the accumulator, each waiting for its own
  entry only. The accumulator ping-pongs between two register sets and is
  back in the first after the batch (K is even). ``acc`` holds the
  accumulator planes in register-slot order; kAccSlot[b] is the slot of plane
  b. Each bounded wait polls at most ``cap`` times; ``gave`` reports a wait
  that gave up.
* ``product_batch(xw, c, wrow, entry)``: the K products of one batch whose
  taps c .. c+K-1 lie in one IFM channel word: all K weight rows are requested
  from the LDS weight ring first (plane b in word kWSlot[b]); per product, bit
  c+k of each IFM word is broadcast into a plane (``v_bfe_i32``), the
  multiplier netlist runs into a register block that holds plane b at
  position kProdSlot[b], and the block goes to this lane's ring entry with
  16-byte stores. Two product blocks alternate, so the stores of one product
  overlap the arithmetic of the next.
* ``product_step(xw, c, wrow, entry)``: the same for one product (batches at a
  channel-word boundary and the last, partial batch).

Port registers are fixed ranges from v96 upwards (from v80, or for the
accumulator from v48, for the widest formats, whose netlists need the room);
the temporaries are the rest of the window up to v255, declared clobbered, so
the compiler's own values stay below or are not live across the blocks.
"""
import re

from .regalloc import AllocError, Block, allocate

BASE = 96
TOP = 256


# Every netlist instruction is an 8-byte VOP3 encoding. Measured on gfx950, a
# run of them issues at 4.04 clocks per instruction when each starts on an
# 8-byte boundary and at 5.04 when each straddles one, so every run starts
# with an alignment directive (the assembler pads with a 4-byte s_nop 0).
ALIGN8 = ".p2align 3"


def lgkm(n):
    """A wait count for s_waitcnt lgkmcnt: the field holds at most 15, and a
    smaller count only waits for more (LDS operations complete in order)."""
    return min(n, 15)


def pad4(n):
    return (n + 3) & ~3


def _rename(lines, mapping):
    pat = re.compile(r"\bv(\d+)\b")
    return [pat.sub(lambda m: f"v{mapping.get(int(m.group(1)), int(m.group(1)))}", ln)
            for ln in lines]


def _asm_string(lines):
    return "\n".join(f'      "{ln}\\n"' for ln in lines)


def split_functions(accum_C, prod_C, nin, nacc, K, slots=2, schedule="batch", sync="barrier",
                    base=None, mul_base=None, top=None):
    """C++ text (inside a variant's namespace) of the two asm functions and
    their slot tables, plus allocation statistics.

    slots: LDS product ring depth (batches in flight; the multiplier runs
    slots-1 batches ahead). schedule: "batch" requests all K entries of a
    batch after its barrier; "step" requests entry k+1 before adding entry k;
    "prefetch" (slots 3) is "step" plus entry 0 of the next batch requested
    before the last add of the current one.

    sync: "barrier" ends every batch with a workgroup barrier; "pairs" hands
    batches over between one accumulator wave and its multiplier wave through
    two LDS counters (at the flag address f: f+0 batches made, f+4 batches
    consumed): before a batch the accumulator reads the counter together with
    the batch's products and uses them if the counter shows the batch (LDS
    operations of a wave complete in order, and the multiplier writes the
    counter after its products); else it polls the counter alone, with a
    sleep between reads, at most `cap` times (a run-time argument), and reads
    the products again; a wait that used up its polls without seeing the
    batch sets `gave` (the caller records it: the results are then invalid).
    After the batch it writes the consumed count. With schedule "early" the
    consumed count is written as soon as the last entry's products are in
    registers, and the counter and entry 0 of the next batch are requested
    before that entry is added, so that the check at the top of the next
    batch finds them arrived."""
    assert slots in (2, 3) and schedule in ("batch", "step", "prefetch", "early")
    assert schedule != "prefetch" or slots == 3
    assert sync in ("barrier", "pairs")
    assert sync == "barrier" or schedule in ("batch", "early")
    assert sync == "pairs" or schedule != "early"
    # first port register of the accumulator's and the multiplier's blocks
    # (the roles are separate branches, so their windows may differ)
    BASE = globals()["BASE"] if base is None else base
    MUL_BASE = BASE if mul_base is None else mul_base
    TOP = globals()["TOP"] if top is None else top  # one past the last register the blocks use
    ninp, naccp = pad4(nin), pad4(nacc)
    kstride = naccp // 4
    A = list(range(BASE, BASE + naccp))
    B = list(range(BASE + naccp, BASE + 2 * naccp))
    P = [list(range(BASE + (2 + k) * naccp, BASE + (3 + k) * naccp)) for k in range(K)]
    VF, VB = TOP - 1, TOP - 2  # flag value read, consumed count written ("pairs")
    pool = list(range(BASE + (2 + K) * naccp, TOP - 2 if sync == "pairs" else TOP))
    lines, place, st_acc = allocate(accum_C, {"acc": Block(A), "p": Block(P[0])},
                                    {"acc": (Block(B), "acc")}, pool)
    acc_slot = [r - BASE for r in place["in"]["acc"]]
    prod_slot = [r - P[0][0] for r in place["in"]["p"]]
    # The ring holds chunk j (16 bytes) of the 64 lanes' entries side by side, so
    # one ds_read_b128 covers 1 KiB without bank conflicts whatever the entry's
    # width (a lane-major layout conflicts when the entry is 4 or 8 chunks).
    chunk_bytes = 64 * 16                # distance between chunks j and j+1
    entry_bytes = 4 * 64 * kstride * 16  # ring distance between batch entries k and k+1
    if (K - 1) * entry_bytes + (kstride - 1) * chunk_bytes > 0xFFFF:
        raise AllocError("product ring offsets exceed the 16-bit LDS offset field")

    def reads(slot, k):
        return [f"ds_read_b128 v[{P[k][4 * j]}:{P[k][4 * j] + 3}], %[e{slot}] "
                f"offset:{k * entry_bytes + chunk_bytes * j}" for j in range(kstride)]

    def netlist(k):
        """Entry k's adder, 8-byte aligned (see ALIGN8)."""
        m = {}
        if k % 2 == 1:  # B -> A
            m.update({a: b for a, b in zip(A, B)})
            m.update({b: a for a, b in zip(A, B)})
        m.update({p0: pk for p0, pk in zip(P[0], P[k])})
        return [ALIGN8] + _rename(lines, m)

    # Events of one batch in issue order: ("r", slot, k) loads entry k of a
    # slot, ("n", k) adds entry k of the current slot.
    def events(slot):
        nxt = (slot + 1) % slots
        ev = []
        if schedule == "batch":
            ev += [("r", slot, k) for k in range(K)]
            ev += [("n", k) for k in range(K)]
        else:
            if schedule == "step":
                ev.append(("r", slot, 0))
            for k in range(K):
                if k + 1 < K:
                    ev.append(("r", slot, k + 1))
                elif schedule == "prefetch":
                    ev.append(("r", nxt, 0))
                ev.append(("n", k))
        return ev

    # The wait before adding entry k leaves in flight only the loads issued
    # after entry k's (LDS operations complete in order). Loads still in
    # flight at a barrier are carried across it ("prefetch" only).
    def pair_batch(slot):
        """One batch handed over through the counters (see sync). The
        counter is read together with the batch's products; if it does not
        show the batch yet, the products are dropped and only the counter is
        read again, after a sleep, until it does (at most `cap` times);
        then the products are read once more."""
        n_reads = K * kstride
        early = schedule == "early"
        if early:
            # the counter and entry 0 were requested during the previous batch
            # (or before the loop); only entry 0's loads were issued after it
            out, ctr_wait = [], kstride
        else:
            out = [f"ds_read_b32 v{VF}, %[fl]"]
            for k in range(K):
                out += reads(slot, k)
            ctr_wait = min(n_reads, 15)
        # the counter is the oldest operation in flight: any count below the
        # loads issued after it (the field holds at most 15) waits for it
        out += [f"s_waitcnt lgkmcnt({ctr_wait})",
                f"v_readfirstlane_b32 %[t], v{VF}",
                "s_nop 4",
                "s_cmp_ge_u32 %[t], %[b1]",
                f"s_cbranch_scc1 L%=_go{slot}",
                "s_waitcnt lgkmcnt(0)",             # batch not made yet: drop the loads
                "s_mov_b32 %[spin], 0",
                f"L%=_poll{slot}:",
                "s_cmp_ge_u32 %[spin], %[cap]",     # the wait's sleeps used up: give up
                f"s_cbranch_scc1 L%=_giveup{slot}",
                "s_sleep 1",
                f"ds_read_b32 v{VF}, %[fl]",
                "s_waitcnt lgkmcnt(0)",
                f"v_readfirstlane_b32 %[t], v{VF}",
                "s_nop 4",
                "s_add_u32 %[spin], %[spin], 1",
                "s_cmp_ge_u32 %[t], %[b1]",
                f"s_cbranch_scc0 L%=_poll{slot}",
                f"s_branch L%=_again{slot}",
                f"L%=_giveup{slot}:",
                "s_mov_b32 %[gave], 1",             # recorded by the caller
                f"L%=_again{slot}:"]
        release = [f"v_mov_b32 v{VB}, %[b1]",
                   "s_nop 4",                      # VALU result -> LDS store data
                   f"ds_write_b32 %[fl], v{VB} offset:4"]
        if early:
            out += reads(slot, 0) + [f"L%=_go{slot}:"]
            for k in range(1, K):
                out += reads(slot, k)
        else:
            for k in range(K):
                out += reads(slot, k)
            out += [f"L%=_go{slot}:"]
        for k in range(K):
            out.append(f"s_waitcnt lgkmcnt({lgkm((K - 1 - k) * kstride)})")
            if early and k == K - 1:
                # every product of this batch is in registers: release the
                # slot, then request the next batch's counter and entry 0
                # (after the last batch they are read and never used)
                out += release + [f"ds_read_b32 v{VF}, %[fl]"] + reads((slot + 1) % slots, 0)
            out += netlist(k)
        if not early:
            out += release
        out += ["s_add_u32 %[b1], %[b1], 1"]
        return out

    if sync == "pairs":
        body = ["s_waitcnt lgkmcnt(0)", "s_mov_b32 %[n], %[nb]", "s_mov_b32 %[b1], 1",
                "s_mov_b32 %[gave], 0"]
        if schedule == "early":
            body += [f"ds_read_b32 v{VF}, %[fl]"] + reads(0, 0)
        body += ["L%=_loop:"]
        for slot in range(slots):
            body += pair_batch(slot)
            body += ["s_sub_u32 %[n], %[n], 1",
                     "s_cmp_eq_u32 %[n], 0",
                     "s_cbranch_scc1 L%=_done"]
        body += ["s_branch L%=_loop", "L%=_done:", "s_waitcnt lgkmcnt(0)"]
        used = set(B) | set(r for blk in P for r in blk) | set(st_acc["temps"]) | {VF, VB}
        clob = ", ".join(f'"v{r}"' for r in sorted(used))
        state = ", ".join(f'"+{{v{BASE + s}}}"(acc[{s}])' for s in range(naccp))
        accum_fn = f"""static constexpr int kAccSlot[{nacc}] = {{{", ".join(map(str, acc_slot))}}};
static constexpr int kProdSlot[{nacc}] = {{{", ".join(map(str, prod_slot))}}};
static constexpr int kSlots = {slots};
static constexpr bool kPairs = true;
// The accumulator role: nb batches of K products from the LDS ring of kSlots
// slots (this lane's first entry of slot s at e_s, batch b in slot b % kSlots),
// handed over by the multiplier wave through the counters at fl (made at fl,
// consumed at fl + 4); acc holds the planes in register-slot order. Each wait
// for a batch sleeps at most cap times; gave is set when one gave up.
static __device__ __forceinline__ void accum_loop(uint32_t (&acc)[{naccp}], const lds_u32* e0,
                                                  const lds_u32* e1, const lds_u32* e2,
                                                  const lds_u32* fl, int nb, uint32_t cap,
                                                  uint32_t& gave) {{
  uint32_t n, b1, spin, t;
  asm volatile(
{_asm_string(body)}
      : {state}, [n] "=&s"(n), [b1] "=&s"(b1), [spin] "=&s"(spin), [t] "=&s"(t),
        [gave] "=&s"(gave)
      : [e0] "v"(e0), [e1] "v"(e1), [e2] "v"(e2), [fl] "v"(fl), [nb] "s"(nb), [cap] "s"(cap)
      : {clob}, "scc", "memory");
}}
"""
        mul_fn, stats = _mul_functions(prod_C, nin, nacc, K, ninp, naccp, kstride, prod_slot,
                                       entry_bytes, st_acc, MUL_BASE, TOP)
        return accum_fn + mul_fn, stats

    carried = [("r", 0, 0)] if schedule == "prefetch" else []
    body = ["s_waitcnt lgkmcnt(0)"]  # nothing of the compiler's in flight: counts below are exact
    if carried:
        body += reads(0, 0)
    body += ["s_mov_b32 %[n], %[nb]", "L%=_loop:"]
    for slot in range(slots):
        inflight = list(carried)
        for e in events(slot):
            if e[0] == "r":
                body += reads(e[1], e[2])
                inflight += [e] * kstride
            else:
                k = e[1]
                last = max(i for i, x in enumerate(inflight) if x == ("r", slot, k))
                newer = len(inflight) - 1 - last
                body.append(f"s_waitcnt lgkmcnt({lgkm(newer)})")
                inflight = inflight[last + 1:]
                body += netlist(k)
        carried = inflight
        body += ["s_barrier",
                 "s_sub_u32 %[n], %[n], 1",
                 "s_cmp_eq_u32 %[n], 0",
                 "s_cbranch_scc1 L%=_done"]
    body += ["s_branch L%=_loop", "L%=_done:", "s_waitcnt lgkmcnt(0)"]
    used = set(B) | set(r for blk in P for r in blk) | set(st_acc["temps"])
    clob = ", ".join(f'"v{r}"' for r in sorted(used))
    state = ", ".join(f'"+{{v{BASE + s}}}"(acc[{s}])' for s in range(naccp))
    accum_fn = f"""static constexpr int kAccSlot[{nacc}] = {{{", ".join(map(str, acc_slot))}}};
static constexpr int kProdSlot[{nacc}] = {{{", ".join(map(str, prod_slot))}}};
static constexpr int kSlots = {slots};
static constexpr bool kPairs = false;
// The accumulator role: nb batches of K products from the LDS ring of kSlots
// slots (this lane's first entry of slot s at e_s, batch b in slot b % kSlots),
// one barrier after each batch; acc holds the planes in register-slot order
// (fl, cap and gave, the pairs' counters and bounded waits, are not used).
static __device__ __forceinline__ void accum_loop(uint32_t (&acc)[{naccp}], const lds_u32* e0,
                                                  const lds_u32* e1, const lds_u32* e2,
                                                  const lds_u32* fl, int nb, uint32_t cap,
                                                  uint32_t& gave) {{
  uint32_t n;
  gave = 0;
  asm volatile(
{_asm_string(body)}
      : {state}, [n] "=&s"(n)
      : [e0] "v"(e0), [e1] "v"(e1), [e2] "v"(e2), [nb] "s"(nb)
      : {clob}, "scc", "memory");
}}
"""
    mul_fn, stats = _mul_functions(prod_C, nin, nacc, K, ninp, naccp, kstride, prod_slot,
                                   entry_bytes, st_acc, MUL_BASE, TOP)
    return accum_fn + mul_fn, stats


def _mul_functions(prod_C, nin, nacc, K, ninp, naccp, kstride, prod_slot, entry_bytes, st_acc,
                   BASE=BASE, TOP=TOP):
    """The multiplier role's asm functions (the same for both sync modes)."""
    # ---- multiplier role: product planes go to the P block in slot order
    # (plane b at word prod_slot[b]), so a product is stored with 16-byte
    # writes; the banks of the product planes are thereby fixed.
    W = [list(range(BASE + k * ninp, BASE + (k + 1) * ninp)) for k in range(K)]
    PB = [list(range(BASE + K * ninp + j * naccp, BASE + K * ninp + (j + 1) * naccp))
          for j in range(2)]
    X = list(range(BASE + K * ninp + 2 * naccp, BASE + K * ninp + 2 * naccp + nin))
    pool2 = list(range(BASE + K * ninp + 2 * naccp + nin, TOP))
    plines, pplace, st_mul = allocate(prod_C, {"w": Block(W[0]), "x": Block(X)},
                                      {"p": [PB[0][0] + prod_slot[b] for b in range(nacc)]}, pool2)
    w_slot = [r - W[0][0] for r in pplace["in"]["w"]]
    xregs = pplace["in"]["x"]

    def mac_section(k, creg, wait):
        """bfe + netlist + stores for product k; `wait` leaves pending only LDS
        operations that neither write row k's weights nor read product
        block k%2."""
        m = {w0: wk for w0, wk in zip(W[0], W[k])}
        m.update({p0: pj for p0, pj in zip(PB[0], PB[k % 2])})
        out = [ALIGN8] + [f"v_bfe_i32 v{r}, %[x{b}], {creg}, 1" for b, r in enumerate(xregs)]
        out.append(f"s_waitcnt lgkmcnt({lgkm(wait)})")
        out += [ALIGN8] + _rename(plines, m)
        out.append("s_nop 4")  # VALU results -> LDS store data
        for j in range(kstride):
            r0 = PB[k % 2][4 * j]
            out.append(f"ds_write_b128 %[e], v[{r0}:{r0 + 3}] "
                       f"offset:{k * entry_bytes + 64 * 16 * j}")
        return out

    nw, np_ = ninp // 4, kstride
    # batch: K weight rows, then K products; LDS operations complete in order
    body2 = []
    for k in range(K):
        for j in range(nw):
            body2.append(f"ds_read_b128 v[{W[k][4 * j]}:{W[k][4 * j] + 3}], %[wr] "
                         f"offset:{k * ninp * 4 + 16 * j}")
    for k in range(K):
        wait = (K - 1 - k) * nw + k * np_      # operations newer than row k's reads
        if k >= 2:
            wait = min(wait, np_)              # product k-2's stores from block k%2 done
        body2 += mac_section(k, f"%[c{k}]", wait)
    # single product (tails and batches that cross a channel word)
    body1 = [f"ds_read_b128 v[{W[0][4 * j]}:{W[0][4 * j] + 3}], %[wr] offset:{16 * j}"
             for j in range(nw)]
    body1 += mac_section(0, "%[c0]", 0)
    used2 = set(r for blk in W for r in blk) | set(r for blk in PB for r in blk) | set(X) | \
        set(st_mul["temps"])
    clob2 = ", ".join(f'"v{r}"' for r in sorted(used2))
    xin = ", ".join(f'[x{b}] "v"(xw[{b}])' for b in range(nin))
    cin = ", ".join(f'[c{k}] "s"(c + {k})' for k in range(K))
    mul_fn = f"""static constexpr int kWSlot[{nin}] = {{{", ".join(map(str, w_slot))}}};
// K products of one batch (taps c .. c+K-1 of one channel word): the weight rows
// from LDS (row k at wrow + k*{ninp} words), bit c+k of each IFM word, the
// multiplier netlist, 16-byte stores to this lane's ring entries.
static __device__ __forceinline__ void product_batch(const uint32_t (&xw)[{nin}], int c,
                                                     const lds_u32* wrow, lds_u32* entry) {{
  asm volatile(
{_asm_string(body2)}
      :
      : {xin}, {cin}, [wr] "v"(wrow), [e] "v"(entry)
      : {clob2}, "memory");
}}
// One product (tap c).
static __device__ __forceinline__ void product_step(const uint32_t (&xw)[{nin}], int c,
                                                    const lds_u32* wrow, lds_u32* entry) {{
  asm volatile(
{_asm_string(body1)}
      :
      : {xin}, [c0] "s"(c), [wr] "v"(wrow), [e] "v"(entry)
      : {clob2}, "memory");
}}
"""
    stats = {"accum": {k: v for k, v in st_acc.items() if k != "temps"},
             "mul": {k: v for k, v in st_mul.items() if k != "temps"}}
    return mul_fn, stats
