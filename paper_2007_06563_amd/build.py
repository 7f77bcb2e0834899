"""Build libhobflops.so: generate the netlists, emit HIP, compile for gfx950.

Steps (the paper's flow, Sec. 3 and its flow figure, with this package's own
tools): build each operator circuit (gen.fp), optimise it and map it onto
3-input LUT cells (gen.opt), emit it as straight-line HIP (gen.emit), then
compile every kernel variant with hipcc for gfx950 and link one shared library
next to this file. Generated sources go to _gen/ (not part of the source tree).
"""
import concurrent.futures as cf
import hashlib
import json
import os
import re
import shlex
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
GEN = os.path.join(HERE, "_gen")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libhobflops.so")
# the VALU issue-rate probe (a diagnostic for the roofline, bench.py --issue-rate)
PROBE_LIB = os.path.join(HERE, "libhobflops_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIPFLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"), "-I", GEN]

if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2007_06563_amd import variants  # noqa: E402
from paper_2007_06563_amd.gen import align, asmgen, banks, emit, fp, opt, regalloc  # noqa: E402


def nb(wE, wF):
    return 3 + wE + wF


def _gen_sources_digest():
    h = hashlib.sha256()
    for name in ("circuit.py", "fp.py", "opt.py", "sim.py", "emit.py", "regalloc.py", "asmgen.py"):
        h.update(open(os.path.join(HERE, "gen", name), "rb").read())
    h.update(open(os.path.abspath(__file__), "rb").read())  # the emission options chosen here
    return h.hexdigest()[:16]


def _circuit_sources_digest():
    """Digest of what the optimised circuits depend on (not their emission)."""
    h = hashlib.sha256()
    for name in ("circuit.py", "fp.py", "opt.py", "sim.py"):
        h.update(open(os.path.join(HERE, "gen", name), "rb").read())
    h.update(repr(_NONCANONICAL).encode())
    h.update(_MAC_RECIPE.encode())
    return h.hexdigest()[:16]


def _circuit_to_json(C):
    return {"name": C.name, "fanins": [list(f) for f in C.fanins], "tts": C.tts,
            "is_input": C.is_input, "inputs": C.inputs, "outputs": C.outputs,
            "input_of": [[n, g, b] for n, (g, b) in C.input_of.items()]}


def _circuit_from_json(d):
    from paper_2007_06563_amd.gen.circuit import Circuit
    C = Circuit(d["name"])
    C.fanins = [tuple(f) for f in d["fanins"]]
    C.tts = list(d["tts"])
    C.is_input = list(d["is_input"])
    C.inputs = [(g, list(l)) for g, l in d["inputs"]]
    C.outputs = [(g, list(l)) for g, l in d["outputs"]]
    C.input_of = {n: (g, b) for n, g, b in d["input_of"]}
    C.table = {(C.tts[n], C.fanins[n]): n for n in range(1, len(C.fanins)) if not C.is_input[n]}
    return C


def _circuit_key(k):
    kind, key, r = k
    return f"{kind}|{','.join(map(str, key))}|{r}"


def _load_circuit_cache():
    """Optimised circuits of earlier builds whose circuit sources are unchanged
    (the optimisation takes minutes; emission and assembly are redone)."""
    path = os.path.join(GEN, "circuits.json")
    if not os.path.exists(path):
        return
    try:
        data = json.load(open(path))
    except (OSError, ValueError):
        return
    if data.get("digest") != _circuit_sources_digest():
        return
    for k, (cj, raw) in data["circuits"].items():
        kind, key, r = k.split("|")
        t = (kind, tuple(int(v) for v in key.split(",")), r)
        if t not in _CIRCUITS:
            _CIRCUITS[t] = (_circuit_from_json(cj), raw)


def _save_circuit_cache():
    path = os.path.join(GEN, "circuits.json")
    data = {"digest": _circuit_sources_digest(),
            "circuits": {_circuit_key(k): [_circuit_to_json(C), raw]
                         for k, (C, raw) in _CIRCUITS.items()}}
    tmp = path + ".tmp"
    with open(tmp, "w") as f:
        json.dump(data, f)
    os.replace(tmp, path)


# Netlists whose results may be non-canonical (they feed only the adder and
# the accumulator), so that E and F of a non-normal result and the sign of a
# NaN are free: the don't-care and resubstitution passes of gen.opt apply to
# them.
_NONCANONICAL = ("accum", "prod")
_CIRCUITS = {}  # (kind, key, rounding name) -> (optimised circuit, raw node count)


# How the fused step's circuit is made (part of the circuit cache's key).
_MAC_RECIPE = ("mac: the smaller of one optimised circuit and product + adder composed; "
               "accum: the smallest of four alignment structures")


def _compose_mac(P, A, key, r):
    """The fused step acc' = A(acc, P(w, x)) built from the optimised product
    and accumulating-adder circuits, with the ports of fp.mac_circuit."""
    from paper_2007_06563_amd.gen.circuit import Circuit
    wE, wi, wa = key
    D = Circuit(fp.mac_circuit(wE, wi, wa, rnd=r).name)
    port = {"acc": D.input("acc", nb(wE, wa)), "w": D.input("w", nb(wE, wi)),
            "x": D.input("x", nb(wE, wi))}

    def place(C, given):
        m = {0: 0}
        for group, lits in C.inputs:
            for l, nl in zip(lits, given[group]):
                m[l >> 1] = nl ^ (l & 1)
        for n in range(1, len(C.fanins)):
            if not C.is_input[n]:
                m[n] = D.lut(C.tts[n], [m[f] for f in C.fanins[n]])
        return {group: [m[l >> 1] ^ (l & 1) for l in lits] for group, lits in C.outputs}

    p = place(P, {"w": port["w"], "x": port["x"]})["p"]
    D.output("acc", place(A, {"acc": port["acc"], "p": p})["acc"])
    return opt.sweep(D)


# The equivalent structures of the accumulating adder (fp.fp_add's late_clear
# and diff_mux); the build keeps the smallest after every pass.
_ACCUM_FORMS = ((True, True), (True, False), (False, True), (False, False))


def _build_circuit(kind, key, r, parts=None, form=None):
    """The operator circuit, optimised and mapped to LUT3 (module level so that
    a process pool can run it). For the fused step, `parts` holds the
    optimised product and adder circuits: their composition (optimised once
    more across the seam) is kept when it is smaller than the step optimised
    as one circuit, which is too wide for the exhaustive passes."""
    if kind == "mac":
        C = fp.mac_circuit(*key, rnd=r)
        if parts is not None:
            raw = C.n_nodes()
            C = opt.optimize(C)
            J = opt.optimize(_compose_mac(*parts, key, r))
            return (J if J.n_nodes() < C.n_nodes() else C), raw
    elif kind == "prod":
        C = fp.product_circuit(*key, rnd=r)
    elif kind == "accum":
        # the equivalent structures of the adder's alignment, each through
        # every pass; the smallest is kept (form: one structure only)
        best = None
        for late_clear, diff_mux in (_ACCUM_FORMS if form is None else [_ACCUM_FORMS[form]]):
            A, raw = _optimise_noncanonical(kind, key, fp.accumulate_circuit(
                *key, rnd=r, late_clear=late_clear, diff_mux=diff_mux))
            if best is None or A.n_nodes() < best[0].n_nodes():
                best = (A, raw)
        return best
    elif kind == "epi":
        wE, wa, wo, act = key
        C = fp.convert_circuit(wE, wa, wo, relu=bool(act), canonical=True, rnd=r)
    elif kind == "scale":
        C = fp.mul_circuit(*key, canonical=True, rnd=r)
    else:
        C = fp.muladd_circuit(*key, rnd=r)
    return _optimise_noncanonical(kind, key, C)


def _optimise_noncanonical(kind, key, C):
    """Optimised and mapped circuit (with the don't-care and resubstitution
    passes for the kinds whose results may be non-canonical), raw size."""
    raw = C.n_nodes()
    C = opt.optimize(C)
    if kind in _NONCANONICAL:
        wE, wFo = key[0], key[-1]
        care = opt.noncanonical_care(wE, wFo)
        D = opt.dont_care_substitute(C, care)
        if D.n_nodes() < C.n_nodes():
            D = opt.optimize(D)
            C = D if D.n_nodes() < C.n_nodes() else C
        D = opt.resubstitute(C, care)
        if D.n_nodes() < C.n_nodes():
            E = opt.optimize(D)
            C = E if E.n_nodes() < D.n_nodes() else D
    return C, raw


def circuit(kind, key, r):
    """Optimised circuit of one operator (memoised per process)."""
    k = (kind, tuple(key), r)
    if k not in _CIRCUITS:
        parts = None
        if kind == "mac":
            wE, wi, wa = key
            parts = (circuit("prod", (wE, wi, wa), r)[0], circuit("accum", (wE, wa), r)[0])
        _CIRCUITS[k] = _build_circuit(kind, key, r, parts)
    return _CIRCUITS[k]


def prepare_circuits(needed, jobs=None):
    """Optimise the circuits in `needed` (kind, key, rounding name) in parallel:
    products and adders first, then the fused steps composed from them."""
    todo = [k for k in dict.fromkeys(needed) if k not in _CIRCUITS]
    if not todo:
        return
    macs = [k for k in todo if k[0] == "mac"]
    first = [k for k in todo if k[0] != "mac"]
    for _, (wE, wi, wa), r in macs:
        first += [k for k in (("prod", (wE, wi, wa), r), ("accum", (wE, wa), r))
                  if k not in _CIRCUITS and k not in first]
    # each adder's structures as jobs of their own, reduced to the smallest
    runs = [(k, None) for k in first if k[0] != "accum"]
    runs += [(k, f) for k in first if k[0] == "accum" for f in range(len(_ACCUM_FORMS))]
    jobs = jobs or min(16, os.cpu_count() or 4)
    with cf.ProcessPoolExecutor(jobs) as ex:
        if runs:
            args = [k + (None, f) for k, f in runs]
            for (k, _), res in zip(runs, ex.map(_build_circuit, *zip(*args))):
                if k not in _CIRCUITS or res[0].n_nodes() < _CIRCUITS[k][0].n_nodes():
                    _CIRCUITS[k] = res
        if macs:
            parts = [(_CIRCUITS[("prod", key, r)][0], _CIRCUITS[("accum", key[::2], r)][0])
                     for _, key, r in macs]
            for k, res in zip(macs, ex.map(_build_circuit, *zip(*macs), parts)):
                _CIRCUITS[k] = res


def _netlist_name(kind, key, rnd):
    """(function name, rounding name) of an operator's netlist."""
    name = {"mac": "mac_e{}m{}_a{}", "epi": "epi_e{}m{}_o{}{}", "muladd": "muladd_e{}m{}_a{}",
            "prod": "prod_e{}m{}_a{}", "accum": "accum_e{}m{}", "scale": "scale_e{}m{}_o{}"}[kind]
    r = variants.RND_NAME[rnd]
    sfx = variants._sfx(rnd)
    if kind == "epi":
        wE, wa, wo, act = key
        # a widening convert rounds nothing: one netlist serves both modes
        if wo >= wa:
            r, sfx = "rne", ""
        return name.format(wE, wa, wo, "_relu" if act else "") + sfx, r
    return name.format(*key) + sfx, r


def netlist(kind, key, rnd, cache):
    """Emitted netlist of one operator (rounding mode rnd: variants.RNE or
    RTZ); cached per generator version."""
    fname, r = _netlist_name(kind, key, rnd)
    if fname in cache:
        return fname, cache[fname]
    C, raw = circuit(kind, key, r)
    text_kw = {"in_place": "acc"} if kind in ("mac", "accum") else {}
    # 8-byte, aligned runs for the fused conv's MAC and the element-wise
    # muladd (measured faster there: first layers 2-6%, wide muladd formats
    # 15-20%); the pooling adder measured 3-4% slower that way
    text_kw["aligned"] = kind in ("mac", "muladd")
    entry = {"text": emit.emit_function(C, fname, **text_kw), "ops": emit.op_count(C),
             "raw_nodes": raw}
    cache[fname] = entry
    return fname, entry


# Product ring depth and load schedule of the split kernel's accumulator role
# (see gen/asmgen.split_functions).
SPLIT_SLOTS, SPLIT_SCHEDULE, SPLIT_SYNC = 2, "batch", "pairs"


# Products per hand-over in the split kernel, in order of preference: the
# largest that keeps the LDS product ring (slots x batch x 256 lanes x entry
# words) within 144 KiB and whose multiplier batch fits the asm registers.
# (Six, where it fits, measured 0.5% slower on the bench layer than four.)
SPLIT_BATCHES = (4, 2)


def split_batches(naccp, slots=None):
    slots = slots or SPLIT_SLOTS
    return [K for K in SPLIT_BATCHES if slots * K * 256 * naccp * 4 <= 144 * 1024]


# The compact form of the split kernel: two workgroups per CU, i.e. two
# accumulator/multiplier wave pairs per SIMD, for launches with between one
# and two chains per SIMD. That needs at most 128 VGPRs a wave (the asm
# blocks end at v128) and an LDS product ring of at most 80 KiB, hence two
# products per hand-over.
COMPACT_TOP, COMPACT_BATCH = 128, 2
COMPACT_BASES = ((32, 48), (24, 48), (32, 56), (24, 40), (32, 40))
# Variants whose compact kernel the compiler could only fit by spilling
# registers to scratch (found by build(), which then rebuilds them without
# the compact form: a spilling kernel would defeat its purpose). The list
# holds for the generator and kernel sources it was found with; after any
# change there every variant is tried in the compact form again.
COMPACT_SPILLS = os.path.join(GEN, "compact_spills.json")


def _compact_digest():
    h = hashlib.sha256(_gen_sources_digest().encode())
    h.update(open(os.path.join(HERE, "csrc", "kernels.hpp"), "rb").read())
    return h.hexdigest()[:16]


def _compact_excluded():
    try:
        d = json.load(open(COMPACT_SPILLS))
    except (OSError, ValueError):
        return set()
    if not isinstance(d, dict) or d.get("digest") != _compact_digest():
        return set()
    return set(d["tags"])


def split_asm(wE, wi, wa, rnd, cache, compact=False):
    """The split kernel's assembly for one variant (with "batch", the products
    per hand-over), or None when the two netlists do not fit the registers the
    asm blocks may use at any batch size. compact: the two-workgroups-per-CU
    form (blocks below v128, two products per hand-over)."""
    key = (f"split_e{wE}m{wi}_a{wa}{variants._sfx(rnd)}"
           f"_s{SPLIT_SLOTS}_{SPLIT_SCHEDULE}_{SPLIT_SYNC}_k" + "".join(map(str, SPLIT_BATCHES)))
    if compact:
        key = f"split_compact_e{wE}m{wi}_a{wa}{variants._sfx(rnd)}_t{COMPACT_TOP}_k{COMPACT_BATCH}"
    if key not in cache:
        r = variants.RND_NAME[rnd]
        nin, nacc = nb(wE, wi), nb(wE, wa)
        acc_c = circuit("accum", (wE, wa), r)[0]
        prod_c = circuit("prod", (wE, wi, wa), r)[0]
        cache[key] = {"text": None, "stats": {"unavailable": "no batch size fits"}}
        # The largest batch that fits; for it, of the asm register windows
        # below, the one with the fewest bank conflicts (more registers let
        # the allocator avoid them), the widest compiler share on a tie. The
        # accumulator's role keeps only a few values of the compiler's, so its
        # window may start as low as v32; the multiplier's stays at v80 or up.
        bases = ((96, 96), (80, 80), (48, 80), (32, 80))
        batches = split_batches(asmgen.pad4(nacc))
        top = None
        if compact:
            bases, batches, top = COMPACT_BASES, [COMPACT_BATCH], COMPACT_TOP
        for K in batches:
            best = None
            for base, mul_base in bases:
                try:
                    text, stats = asmgen.split_functions(acc_c, prod_c, nin, nacc, K,
                                                         SPLIT_SLOTS, SPLIT_SCHEDULE, SPLIT_SYNC,
                                                         base=base, mul_base=mul_base, top=top)
                except regalloc.AllocError as e:
                    cache[key] = {"text": None, "stats": {"unavailable": str(e)}}
                    continue
                cost = (stats["accum"]["conflicts"] + stats["accum"]["off_bank"]
                        + stats["mul"]["conflicts"] + stats["mul"]["off_bank"])
                if best is None or cost < best[0]:
                    stats["batch"], stats["base"] = K, [base, mul_base]
                    best = (cost, text, stats)
            if best is not None:
                cache[key] = {"text": best[1], "stats": best[2], "batch": K}
                break
    return cache[key] if cache[key]["text"] is not None else None


def generate(verbose=True):
    os.makedirs(GEN, exist_ok=True)
    compact_excluded = _compact_excluded()
    digest = _gen_sources_digest()
    cache_path = os.path.join(GEN, "netlists.json")
    cache = {}
    if os.path.exists(cache_path):
        data = json.load(open(cache_path))
        if data.get("digest") == digest:
            cache = data["netlists"]
    files = []
    reg_conv, reg_mul = [], []
    # every circuit whose netlist or split assembly is not cached, optimised in
    # parallel first
    needed = []
    for wE, wi, wa, wo, act, rnd in variants.CONV_VARIANTS:
        r = variants.RND_NAME[rnd]
        for kind, key in (("mac", (wE, wi, wa)), ("epi", (wE, wa, wo, act)),
                          ("prod", (wE, wi, wa)), ("accum", (wE, wa))):
            fname, rr = _netlist_name(kind, key, rnd)
            if fname not in cache:
                needed.append((kind, key, rr))
        skey = (f"split_e{wE}m{wi}_a{wa}{variants._sfx(rnd)}"
                f"_s{SPLIT_SLOTS}_{SPLIT_SCHEDULE}_{SPLIT_SYNC}_k" + "".join(map(str, SPLIT_BATCHES)))
        if skey not in cache:
            needed += [("accum", (wE, wa), r), ("prod", (wE, wi, wa), r)]
    for wE, wi, wa, rnd in variants.MULADD_VARIANTS:
        if _netlist_name("muladd", (wE, wi, wa), rnd)[0] not in cache:
            needed.append(("muladd", (wE, wi, wa), variants.RND_NAME[rnd]))
    for wE, wi, wa, wo, rnd in variants.POOL_VARIANTS:
        for kind, key in (("accum", (wE, wa)), ("scale", (wE, wa, wo))):
            fname, rr = _netlist_name(kind, key, rnd)
            if fname not in cache:
                needed.append((kind, key, rr))
    _load_circuit_cache()
    prepare_circuits(needed)
    _save_circuit_cache()
    for v in variants.CONV_VARIANTS:
        wE, wi, wa, wo, act, rnd = v
        tag = variants.conv_tag(v)
        mac, mac_e = netlist("mac", (wE, wi, wa), rnd, cache)
        epi, _ = netlist("epi", (wE, wa, wo, act), rnd, cache)
        prod, prod_e = netlist("prod", (wE, wi, wa), rnd, cache)
        accum, accum_e = netlist("accum", (wE, wa), rnd, cache)
        sp = split_asm(wE, wi, wa, rnd, cache)
        split_text = sp["text"] if sp else ""
        spc = (split_asm(wE, wi, wa, rnd, cache, compact=True)
               if sp and f"conv_{tag}" not in compact_excluded else None)
        compact_text = f"namespace compact {{\n{spc['text']}}}  // namespace compact\n" if spc else ""
        split_members = """  static constexpr int kBatch = {batch};
  static constexpr const int* kAccSlot = conv_{tag}::kAccSlot;
  static constexpr const int* kProdSlot = conv_{tag}::kProdSlot;
  static constexpr const int* kWSlot = conv_{tag}::kWSlot;
  static constexpr int kSlots = conv_{tag}::kSlots;
  static constexpr bool kPairs = conv_{tag}::kPairs;
  static __device__ __forceinline__ void accum_loop(uint32_t (&acc)[(NACC + 3) & ~3],
                                                    const lds_u32* e0, const lds_u32* e1,
                                                    const lds_u32* e2, const lds_u32* fl,
                                                    int nb, uint32_t cap, uint32_t& gave) {{
    conv_{tag}::accum_loop(acc, e0, e1, e2, fl, nb, cap, gave);
  }}
  static __device__ __forceinline__ void product_step(const uint32_t (&xw)[NIN], int c,
                                                      const lds_u32* wrow, lds_u32* entry) {{
    conv_{tag}::product_step(xw, c, wrow, entry);
  }}
  static __device__ __forceinline__ void product_batch(const uint32_t (&xw)[NIN], int c,
                                                       const lds_u32* wrow, lds_u32* entry) {{
    conv_{tag}::product_batch(xw, c, wrow, entry);
  }}
""".format(batch=sp["batch"], tag=tag) if sp else ""
        # the compact form: the same kernel body with the compact asm blocks
        compact_struct = """struct VC : V {{
  static constexpr int kBatch = {batch};
  static constexpr const int* kAccSlot = compact::kAccSlot;
  static constexpr const int* kProdSlot = compact::kProdSlot;
  static constexpr const int* kWSlot = compact::kWSlot;
  static constexpr int kSlots = compact::kSlots;
  static constexpr bool kPairs = compact::kPairs;
  static __device__ __forceinline__ void accum_loop(uint32_t (&acc)[(NACC + 3) & ~3],
                                                    const lds_u32* e0, const lds_u32* e1,
                                                    const lds_u32* e2, const lds_u32* fl,
                                                    int nb, uint32_t cap, uint32_t& gave) {{
    compact::accum_loop(acc, e0, e1, e2, fl, nb, cap, gave);
  }}
  static __device__ __forceinline__ void product_step(const uint32_t (&xw)[NIN], int c,
                                                      const lds_u32* wrow, lds_u32* entry) {{
    compact::product_step(xw, c, wrow, entry);
  }}
  static __device__ __forceinline__ void product_batch(const uint32_t (&xw)[NIN], int c,
                                                       const lds_u32* wrow, lds_u32* entry) {{
    compact::product_batch(xw, c, wrow, entry);
  }}
}};
""".format(batch=spc["batch"]) if spc else ""
        split_launch = (f"""  if (algo == kAlgoSplitCompact)
    hipLaunchKernelGGL(conv2d_split_compact_kernel<conv_{tag}::VC>, grid, dim3(2 * kConvBlock), 0,
                       stream, ifm, w, ofm, p);
  else
""" if spc else "") + (f"""  if (algo == kAlgoSplit)
    hipLaunchKernelGGL(conv2d_split_kernel<conv_{tag}::V>, grid, dim3(2 * kConvBlock), 0, stream,
                       ifm, w, ofm, p);
  else
""" if sp else "")
        src = f"""// Generated: convolution variant {tag}. Do not edit.
#include "kernels.hpp"
#include "registry.hpp"
namespace hobflops {{
namespace conv_{tag} {{
{cache[mac]['text']}
{cache[epi]['text']}
{cache[prod]['text']}
{cache[accum]['text']}
{split_text}
{compact_text}
struct V {{
  static constexpr int NIN = {nb(wE, wi)}, NACC = {nb(wE, wa)}, NOUT = {nb(wE, wo)};
  static constexpr int wE = {wE}, wF_OUT = {wo};
{split_members}  static __device__ __forceinline__ void mac(uint32_t (&acc)[NACC], const uint32_t (&w)[NIN],
                                             const uint32_t (&x)[NIN]) {{ {mac}(acc, w, x); }}
  static __device__ __forceinline__ void mul(const uint32_t (&w)[NIN], const uint32_t (&x)[NIN],
                                             uint32_t (&p)[NACC]) {{ {prod}(w, x, p); }}
  static __device__ __forceinline__ void add(uint32_t (&acc)[NACC], const uint32_t (&p)[NACC]) {{
    {accum}(acc, p);
  }}
  static __device__ __forceinline__ void epi(const uint32_t (&acc)[NACC], uint32_t (&out)[NOUT]) {{
    {epi}(acc, out);
  }}
}};
{compact_struct}}}  // namespace conv_{tag}
hipError_t launch_conv_{tag}(const uint32_t* ifm, const uint32_t* w, uint32_t* ofm,
                              const ConvParams& p, int algo, hipStream_t stream) {{
  dim3 grid((unsigned)((p.P + kConvBlock - 1) / kConvBlock), (unsigned)p.MT);
{split_launch}    hipLaunchKernelGGL(conv2d_kernel<conv_{tag}::V>, grid, dim3(kConvBlock), 0, stream, ifm, w, ofm, p);
  return hipGetLastError();
}}
}}  // namespace hobflops
"""
        files.append((f"conv_{tag}.hip", src))
        reg_conv.append((v, tag, mac_e["ops"], prod_e["ops"], accum_e["ops"], 1 if sp else 0,
                         1 if spc else 0))
    for v in variants.MULADD_VARIANTS:
        wE, wi, wa, rnd = v
        tag = variants.muladd_tag(v)
        fn, e = netlist("muladd", (wE, wi, wa), rnd, cache)
        src = f"""// Generated: element-wise MAC variant {tag}. Do not edit.
#include "kernels.hpp"
#include "registry.hpp"
namespace hobflops {{
namespace muladd_{tag} {{
{cache[fn]['text']}
struct V {{
  static constexpr int NIN = {nb(wE, wi)}, NACC = {nb(wE, wa)};
  static __device__ __forceinline__ void muladd(const uint32_t (&a)[NIN], const uint32_t (&b)[NIN],
                                                const uint32_t (&c)[NIN], uint32_t (&r)[NACC]) {{
    {fn}(a, b, c, r);
  }}
}};
}}  // namespace muladd_{tag}
hipError_t launch_muladd_{tag}(const uint32_t* a, const uint32_t* b, const uint32_t* c,
                                uint32_t* r, int64_t groups, hipStream_t stream) {{
  const unsigned blocks = (unsigned)((groups + 255) / 256);
  hipLaunchKernelGGL(muladd_kernel<muladd_{tag}::V>, dim3(blocks), dim3(256), 0, stream, a, b, c, r, groups);
  return hipGetLastError();
}}
}}  // namespace hobflops
"""
        files.append((f"muladd_{tag}.hip", src))
        reg_mul.append((v, tag, e["ops"]))
    reg_pool = []
    for v in variants.POOL_VARIANTS:
        wE, wi, wa, wo, rnd = v
        tag = variants.pool_tag(v)
        accum, accum_e = netlist("accum", (wE, wa), rnd, cache)
        scale, scale_e = netlist("scale", (wE, wa, wo), rnd, cache)
        src = f"""// Generated: global average pooling variant {tag}. Do not edit.
#include "kernels.hpp"
#include "registry.hpp"
namespace hobflops {{
namespace pool_{tag} {{
{cache[accum]['text']}
{cache[scale]['text']}
struct V {{
  static constexpr int NIN = {nb(wE, wi)}, NACC = {nb(wE, wa)}, NOUT = {nb(wE, wo)};
  static __device__ __forceinline__ void add(uint32_t (&acc)[NACC], const uint32_t (&x)[NACC]) {{
    {accum}(acc, x);
  }}
  static __device__ __forceinline__ void scale(const uint32_t (&acc)[NACC], const uint32_t (&s)[NACC],
                                               uint32_t (&out)[NOUT]) {{
    {scale}(acc, s, out);
  }}
}};
}}  // namespace pool_{tag}
hipError_t launch_pool_{tag}(const uint32_t* in, uint32_t* out, const PoolParams& p,
                              hipStream_t stream) {{
  const int64_t lanes = (int64_t)p.N * p.CG;
  hipLaunchKernelGGL(avgpool_kernel<pool_{tag}::V>, dim3((unsigned)((lanes + 255) / 256)), dim3(256),
                     0, stream, in, out, p);
  return hipGetLastError();
}}
}}  // namespace hobflops
"""
        files.append((f"pool_{tag}.hip", src))
        reg_pool.append((v, tag, accum_e["ops"], scale_e["ops"]))
    reg = ["// Generated: table of kernel variants (host code). Do not edit.",
           '#include "registry.hpp"', "#ifndef __HIP_DEVICE_COMPILE__", "namespace hobflops {"]
    for v, tag, *_ in reg_conv:
        reg.append(f"hipError_t launch_conv_{tag}(const uint32_t*, const uint32_t*, uint32_t*, "
                   f"const ConvParams&, int, hipStream_t);")
    for v, tag, ops in reg_mul:
        reg.append(f"hipError_t launch_muladd_{tag}(const uint32_t*, const uint32_t*, const uint32_t*, "
                   f"uint32_t*, int64_t, hipStream_t);")
    for v, tag, *_ in reg_pool:
        reg.append(f"hipError_t launch_pool_{tag}(const uint32_t*, uint32_t*, const PoolParams&, "
                   f"hipStream_t);")
    reg.append("const ConvVariant kConvVariants[] = {")
    for v, tag, ops, pops, aops, has_split, has_compact in reg_conv:
        reg.append(f"  {{{v[0]}, {v[1]}, {v[2]}, {v[3]}, {v[4]}, {v[5]}, {has_split}, "
                   f"{has_compact}, {ops}, {pops}, {aops}, launch_conv_{tag}}},")
    reg.append("};")
    reg.append(f"const int kNumConvVariants = {len(reg_conv)};")
    reg.append("const MuladdVariant kMuladdVariants[] = {")
    for v, tag, ops in reg_mul:
        reg.append(f"  {{{v[0]}, {v[1]}, {v[2]}, {v[3]}, {ops}, launch_muladd_{tag}}},")
    reg.append("};")
    reg.append(f"const int kNumMuladdVariants = {len(reg_mul)};")
    reg.append("const PoolVariant kPoolVariants[] = {")
    for v, tag, aops, sops in reg_pool:
        reg.append(f"  {{{v[0]}, {v[1]}, {v[2]}, {v[3]}, {v[4]}, {aops}, {sops}, launch_pool_{tag}}},")
    reg.append("};")
    reg.append(f"const int kNumPoolVariants = {len(reg_pool)};")
    reg.append("}  // namespace hobflops")
    reg.append("#endif")
    files.append(("registry.hip", "\n".join(reg) + "\n"))
    for name, text in files:
        path = os.path.join(GEN, name)
        if not os.path.exists(path) or open(path).read() != text:
            with open(path, "w") as f:
                f.write(text)
    json.dump({"digest": digest, "netlists": cache}, open(cache_path, "w"))
    gates = {k: ({"ops": e["ops"], "raw_nodes": e["raw_nodes"]} if "ops" in e else e["stats"])
             for k, e in cache.items()}
    json.dump(gates, open(os.path.join(GEN, "gates.json"), "w"), indent=1, sort_keys=True)
    if verbose:
        for k in sorted(gates):
            g = gates[k]
            if "ops" in g:
                print(f"  {k}: {g['ops']} ops (raw {g['raw_nodes']})")
            elif "unavailable" in g:
                print(f"  {k}: no split kernel ({g['unavailable']})")
            else:
                print(f"  {k}: accum {g['accum']}, mul {g['mul']}")
    return [os.path.join(GEN, n) for n, _ in files]


LLVM_MC = "/opt/rocm/llvm/bin/llvm-mc"
# Kernels the alignment pass is applied to (mangled names, as in the code
# section names): measured faster with it (element-wise muladd up to 11 %,
# pooling 5 %) or no slower. The fused conv and the unpack kernel run many
# waves per SIMD, which hide a wave's misaligned fetches, and measured up to
# 5 % slower with the pass's re-encodings and nops; they are left as compiled.
ALIGN_KERNELS = ("19conv2d_split_kernel", "13muladd_kernel", "14avgpool_kernel", "11pack_kernel")
# Kernels whose compiled netlists get the VGPR bank pass (gen/banks.py): the
# fused conv, whose MAC runs with several waves per SIMD, where an
# instruction reading two sources from one bank costs about twice the time.
BANK_KERNELS = ("13conv2d_kernel",)


def _compile_plain(src, obj):
    cmd = [HIPCC] + HIPFLAGS + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr[-4000:]}")
    return obj


def _compact_spills(text):
    """Variant tags whose compact split kernel uses scratch (spilled VGPRs),
    from the kernel descriptors of one source's device assembly."""
    out = []
    for m in re.finditer(r"\.amdhsa_kernel (\S+)\n((?:\s+\.amdhsa\w+ [^\n]*\n)+)", text):
        name, body = m.group(1), m.group(2)
        k = name.find("27conv2d_split_compact_kernelINS_")
        seg = re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", body)
        if k < 0 or not seg or int(seg.group(1)) == 0:
            continue
        rest = name[k + len("27conv2d_split_compact_kernelINS_"):]
        n = re.match(r"\d+", rest)
        out.append(rest[n.end():n.end() + int(n.group(0))])
    return out


def _compile(src, obj, stats=None):
    """hipcc -c, with the device code taken through assembly text so that
    gen/align.py can keep its 8-byte instructions 8-byte aligned: the
    driver's own steps (hipcc -###) are run one by one, the device step
    writing assembly instead of an object, which is aligned and assembled
    into the object the later steps (link, bundle, host compile) expect."""
    r = subprocess.run([HIPCC, "-###"] + HIPFLAGS + ["-c", src, "-o", obj],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -### failed on {src}:\n{r.stderr[-4000:]}")
    cmds = [shlex.split(line) for line in r.stderr.splitlines() if line.startswith(' "')]
    dev = [c for c in cmds if "-fcuda-is-device" in c and "-emit-obj" in c]
    if len(dev) != 1:
        raise RuntimeError(f"unexpected hipcc pipeline for {src}: {len(dev)} device steps")
    dev = dev[0]
    k = dev.index("-o")
    dev_obj = dev[k + 1]
    asm, fixed = obj + ".dev.s", obj + ".dev.aligned.s"
    to_asm = list(dev)
    to_asm[to_asm.index("-emit-obj")] = "-S"
    to_asm[k + 1] = asm
    temps = [asm, fixed] + [c[c.index("-o") + 1] for c in cmds if "-o" in c and c is not cmds[-1]]
    temps += [a.split("=", 1)[1] for c in cmds for a in c if a.startswith("-output=")]
    try:
        for c in cmds:
            if c is dev:
                r = subprocess.run(to_asm, capture_output=True, text=True)
                if r.returncode != 0:
                    raise RuntimeError(f"device compile failed on {src}:\n{r.stderr[-4000:]}")
                text = open(asm).read()
                spills = _compact_spills(text)
                text, bst = banks.rename_text(text, only=BANK_KERNELS)
                if bst["blocks"]:
                    with open(asm, "w") as f:
                        f.write(text)
                new, st = align.align_text(text, align.encoding_sizes(asm, LLVM_MC),
                                           only=ALIGN_KERNELS)
                st.update({k: v for k, v in bst.items() if k.startswith("conflicts")})
                st["compact_spills"] = spills
                with open(fixed, "w") as f:
                    f.write(new)
                c = [LLVM_MC, "-triple=amdgcn-amd-amdhsa", "-mcpu=gfx950", "-filetype=obj",
                     "-o", dev_obj, fixed]
                if stats is not None:
                    stats[os.path.basename(src)] = st
            r = subprocess.run(c, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"{os.path.basename(c[0])} failed on {src}:\n"
                                   f"{r.stderr[-4000:]}")
    finally:
        for t in temps:
            if t != obj and os.path.exists(t):
                os.remove(t)
    return obj


def build(jobs=None, verbose=True):
    """Generate and compile everything; returns the library path."""
    gen_files = generate(verbose=verbose)
    srcs = [os.path.join(HERE, "csrc", "abi.hip"), os.path.join(HERE, "csrc", "pack.hip")] + gen_files
    os.makedirs(OBJ, exist_ok=True)
    jobs = jobs or min(16, os.cpu_count() or 4)
    stats = {}

    def compile_all(files):
        with cf.ThreadPoolExecutor(jobs) as ex:
            futs = [ex.submit(_compile, f, os.path.join(OBJ, os.path.basename(f) + ".o"), stats)
                    for f in files]
            return [f.result() for f in futs]

    objs = compile_all(srcs)
    spilled = sorted({t for st in stats.values() for t in st.get("compact_spills", [])})
    if spilled:
        # drop the compact form of those variants and compile their sources again
        json.dump({"digest": _compact_digest(),
                   "tags": sorted(_compact_excluded() | set(spilled))}, open(COMPACT_SPILLS, "w"))
        if verbose:
            print("compact split kernel spills registers, left out:", ", ".join(spilled))
        generate(verbose=False)
        compile_all([os.path.join(GEN, t + ".hip") for t in spilled] +
                    [os.path.join(GEN, "registry.hip")])
    if verbose:
        tot = {k: sum(st.get(k, 0) for st in stats.values())
               for k in ("promoted", "nops", "left", "conflicts_before", "conflicts_after")}
        print(f"8-byte alignment: {tot['promoted']} VALU instructions re-encoded as VOP3, "
              f"{tot['nops']} s_nop inserted, {tot['left']} short runs left")
        print(f"VGPR banks: {tot['conflicts_before']} -> {tot['conflicts_after']} instructions "
              "with two sources in one bank in the renamed blocks")
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-4000:]}")
    os.replace(tmp, LIB)
    # the probe's misaligned streams are deliberate: no alignment pass
    probe_obj = _compile_plain(os.path.join(HERE, "csrc", "issue_probe.hip"),
                               os.path.join(OBJ, "issue_probe.hip.o"))
    tmp = PROBE_LIB + ".tmp"
    r = subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp, probe_obj],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-4000:]}")
    os.replace(tmp, PROBE_LIB)
    if verbose:
        print("built", LIB, "and", PROBE_LIB)
    return LIB


if __name__ == "__main__":
    build()
