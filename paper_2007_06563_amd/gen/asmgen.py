"""Inline-assembly device functions for the split convolution kernel.

The two wave roles of the split kernel run their netlists as inline assembly
with explicit registers chosen by gen.regalloc, so that no VALU instruction
reads two VGPRs of one bank (see gen/regalloc.py). The functions produced:

* ``accum_loop(acc, e0, e1, e2, nb)``: the whole accumulator role. Batch b
  (K products) sits in slot b % kSlots of the LDS product ring; its entries
  are requested with 16-byte loads at immediate offsets from this lane's first
  entry, on the schedule split_functions is given, and K copies of the adder
  netlist add them into the accumulator, each waiting for its own entry only.
  The accumulator ping-pongs between two register sets and is back in the
  first after the batch (K is even). ``acc`` holds the accumulator planes in
  register-slot order; kAccSlot[b] is the slot of plane b.
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

Port registers are fixed ranges from v96 upwards; the temporaries are the
rest of v96..v255, declared clobbered, so the compiler's own values stay below
or are not live across the blocks.
"""
import re

from .regalloc import Block, allocate

BASE = 96
TOP = 256


def pad4(n):
    return (n + 3) & ~3


def _rename(lines, mapping):
    pat = re.compile(r"\bv(\d+)\b")
    return [pat.sub(lambda m: f"v{mapping.get(int(m.group(1)), int(m.group(1)))}", ln)
            for ln in lines]


def _asm_string(lines):
    return "\n".join(f'      "{ln}\\n"' for ln in lines)


def split_functions(accum_C, prod_C, nin, nacc, K, slots=2, schedule="batch"):
    """C++ text (inside a variant's namespace) of the two asm functions and
    their slot tables, plus allocation statistics.

    slots: LDS product ring depth (batches in flight; the multiplier runs
    slots-1 batches ahead). schedule: "batch" requests all K entries of a
    batch after its barrier; "step" requests entry k+1 before adding entry k;
    "prefetch" (slots 3) is "step" plus entry 0 of the next batch requested
    before the last add of the current one."""
    assert slots in (2, 3) and schedule in ("batch", "step", "prefetch")
    assert schedule != "prefetch" or slots == 3
    ninp, naccp = pad4(nin), pad4(nacc)
    kstride = naccp // 4
    A = list(range(BASE, BASE + naccp))
    B = list(range(BASE + naccp, BASE + 2 * naccp))
    P = [list(range(BASE + (2 + k) * naccp, BASE + (3 + k) * naccp)) for k in range(K)]
    pool = list(range(BASE + (2 + K) * naccp, TOP))
    lines, place, st_acc = allocate(accum_C, {"acc": Block(A), "p": Block(P[0])},
                                    {"acc": (Block(B), "acc")}, pool)
    acc_slot = [r - BASE for r in place["in"]["acc"]]
    prod_slot = [r - P[0][0] for r in place["in"]["p"]]
    entry_bytes = 4 * 64 * kstride * 16  # ring distance between batch entries k and k+1

    def reads(slot, k):
        return [f"ds_read_b128 v[{P[k][4 * j]}:{P[k][4 * j] + 3}], %[e{slot}] "
                f"offset:{k * entry_bytes + 16 * j}" for j in range(kstride)]

    def netlist(k):
        m = {}
        if k % 2 == 1:  # B -> A
            m.update({a: b for a, b in zip(A, B)})
            m.update({b: a for a, b in zip(A, B)})
        m.update({p0: pk for p0, pk in zip(P[0], P[k])})
        return _rename(lines, m)

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
                body.append(f"s_waitcnt lgkmcnt({newer})")
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
// The accumulator role: nb batches of K products from the LDS ring of kSlots
// slots (this lane's first entry of slot s at e_s, batch b in slot b % kSlots),
// one barrier after each batch; acc holds the planes in register-slot order.
static __device__ __forceinline__ void accum_loop(uint32_t (&acc)[{naccp}], const lds_u32* e0,
                                                  const lds_u32* e1, const lds_u32* e2, int nb) {{
  uint32_t n;
  asm volatile(
{_asm_string(body)}
      : {state}, [n] "=&s"(n)
      : [e0] "v"(e0), [e1] "v"(e1), [e2] "v"(e2), [nb] "s"(nb)
      : {clob}, "scc", "memory");
}}
"""
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
        out = [f"v_bfe_i32 v{r}, %[x{b}], {creg}, 1" for b, r in enumerate(xregs)]
        out.append(f"s_waitcnt lgkmcnt({wait})")
        out += _rename(plines, m)
        out.append("s_nop 4")  # VALU results -> LDS store data
        for j in range(kstride):
            r0 = PB[k % 2][4 * j]
            out.append(f"ds_write_b128 %[e], v[{r0}:{r0 + 3}] offset:{k * entry_bytes + 16 * j}")
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
    return accum_fn + mul_fn, stats
