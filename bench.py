#!/usr/bin/env python3
"""Benchmark of the HOBFLOPS MCMK convolution on one MI355X.

Workload: the ResNet-shaped layer 8x56x56x64 -> 64 kernels 3x3, stride 1,
pad 1, inputs rounded to the 9-bit format (wE, wF) = (5, 3), multiply and
accumulate in (5, 4) (the paper's HOBFLOPS9 MAC), fixed accumulation order
(ky, kx, c). One step is the whole path on one batch: quantise + pack the
float32 IFM and weights into bit-planes, then the bitsliced convolution, whose
epilogue writes the OFM as float32 (the unpack fused in). Inputs are
synthetic, seeded, resident in HBM before timing starts.

Prints one JSON line: GMAC/s of the step, the convolution kernel against the
VALU roofline (achieved 32-bit bitwise VALU lane-ops/s from the generated
netlist's instruction count and the kernel's HIP-event time), and the CPU
oracle timed on a bounded sample of the same outputs.
"""
import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2007_06563_amd import hobflops as hf  # noqa: E402
from paper_2007_06563_amd import inputs as I     # noqa: E402

# MI355X: 256 CUs of 4 SIMDs at up to 2.4 GHz. A SIMD retires 32 lanes of a
# 32-bit VALU op per clock (128 lanes/clk/CU: the unit rate behind the
# 157.3 TFLOP/s FP32-vector figure, one FMA = 2 flops), but one wave issues at
# most one instruction every 4 clocks, i.e. half a SIMD: two or more waves per
# SIMD are needed to reach the peak.
N_CU, LANES_PER_CU_CLK, CLOCK_HZ = 256, 128, 2.4e9
PEAK_LANE_OPS = N_CU * LANES_PER_CU_CLK * CLOCK_HZ   # 7.86e13 32-bit VALU ops/s
N_SIMD = N_CU * 4
HBM_PEAK = 8.0e12
# clocks per instruction of one wave with a SIMD to itself (measured on MI355X
# with the split kernel's accumulator loop alone in the kernel, shader-clock
# stamps around the loop: 4.44; the issue-rate probe's aligned 8-byte
# v_bitop3_b32 stream: 4.26 including its loop branch), and of a SIMD shared
# by two or more waves of bank-conflict-free bitwise instructions (probe:
# 2.10-2.13; in kernels 2.2-2.4: the peak assumes 2)
ISSUE_CLOCKS = 4.44
SIMD_CLOCKS = 2.24

IN_FMT, ACC_FMT, OUT_FMT = (5, 3), (5, 4), (5, 4)

# HBM bytes per launch of the convolution kernel from rocprofv3 --pmc
# FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what the same
# counter reads for a plain 256 MiB device copy (FETCH x2.0, WRITE x1.0); see
# the profiles/ summaries. Set to None whenever the kernel changes, until the
# counters are taken again.
TRAFFIC = (3552.3 * 2.0 + 6276.3 * 1.0) * 1024   # 13.70 MB (split kernel, float32 OFM)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(ifm, w, s, gpu_codes, seconds):
    """The oracle on a bounded random sample of the layer's outputs, all host
    threads; also its output compared with the GPU's at those points."""
    import oracle
    t = time.perf_counter()
    qi = oracle.quantize_f32(ifm, *IN_FMT)
    qw = oracle.quantize_f32(w, *IN_FMT)
    log(f"cpu_baseline: quantised inputs in {time.perf_counter() - t:.1f}s")
    g = np.random.default_rng(2024)
    threads = oracle.default_threads()
    taps = s.KH * s.KW * s.C

    def pts_of(n):
        return np.stack([g.integers(0, s.N, n), g.integers(0, s.OH, n), g.integers(0, s.OW, n),
                         g.integers(0, s.M, n)], 1).astype(np.int64)

    probe = pts_of(max(64, threads * 8))
    t = time.perf_counter()
    oracle.conv2d_points(qi, qw, probe, s.stride, s.pad, IN_FMT[0], IN_FMT[1], ACC_FMT[1],
                         OUT_FMT[1], nthreads=threads)
    rate = len(probe) / max(time.perf_counter() - t, 1e-6)
    npts = int(min(max(rate * seconds, 256), s.N * s.OH * s.OW * s.M))
    pts = pts_of(npts)
    t = time.perf_counter()
    out = oracle.conv2d_points(qi, qw, pts, s.stride, s.pad, IN_FMT[0], IN_FMT[1], ACC_FMT[1],
                               OUT_FMT[1], nthreads=threads)
    dt = time.perf_counter() - t
    mism = int(np.count_nonzero(out != gpu_codes[pts[:, 0], pts[:, 1], pts[:, 2], pts[:, 3]]))
    # one thread, smaller sample, for comparison with single-core figures
    p1 = pts_of(max(32, npts // threads // 4))
    t = time.perf_counter()
    oracle.conv2d_points(qi, qw, p1, s.stride, s.pad, IN_FMT[0], IN_FMT[1], ACC_FMT[1],
                         OUT_FMT[1], nthreads=1)
    dt1 = time.perf_counter() - t
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": npts * taps / dt / 1e9, "unit": "GMAC/s", "cores": threads, "kind": "oracle",
        "sample": f"{npts} random outputs of {s.N * s.OH * s.OW * s.M} ({npts * taps} MACs) of "
                  f"the same layer, {threads} threads over outputs, {dt:.1f}s",
        "value_1thread": len(p1) * taps / dt1 / 1e9, "cpu_model": cpu,
        "parity_sample_mismatches": mism, "parity_sample_points": npts,
    }


def _time(fn, reps, stream):
    """Average ms of fn() over reps launches (HIP events on the stream)."""
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


KERNEL_NAME = {1: "fused", 2: "split", 3: "split_compact"}


def _conv_ops(d):
    """(kernel shape the library runs d in, VALU ops per 32-MAC word of that
    kernel)."""
    algo = hf.conv2d_algo(d)
    ops = hf.netlist_ops((d.in_fmt.wE, d.in_fmt.wF), (d.acc_fmt.wE, d.acc_fmt.wF), d.round)
    return algo, (ops["mac"] if algo == hf.ALGO_FUSED else ops["mul"] + ops["accum"])


def issue_ceiling(d, algo):
    """The share of the VALU peak a convolution launch can reach, from its
    structure at the nominal clock: every output is one chain of taps in a
    fixed order, and a wave issues at most one instruction per ISSUE_CLOCKS.
    Split kernel: one accumulator wave per chain set, on a SIMD of its own, so
    the time is at least taps x adder instructions x ISSUE_CLOCKS. Fused
    kernel: a wave's taps x MAC instructions x ISSUE_CLOCKS, or its SIMD's
    share of all waves x SIMD_CLOCKS per instruction when several share one
    (workgroups of four waves spread over a CU's four SIMDs)."""
    OH, OW = hf.conv_out_hw(d)
    P, taps = d.N * OH * OW, d.KH * d.KW * d.C
    chain_waves = ((P + 63) // 64) * ((d.M + 31) // 32)
    ops = hf.netlist_ops((d.in_fmt.wE, d.in_fmt.wF), (d.acc_fmt.wE, d.acc_fmt.wF), d.round)
    if algo == hf.ALGO_SPLIT:
        G, clocks = ops["mul"] + ops["accum"], taps * ops["accum"] * ISSUE_CLOCKS
        if chain_waves > N_SIMD:  # more chain sets than SIMDs: some run one after another
            clocks *= -(-chain_waves // N_SIMD)
    elif algo == hf.ALGO_SPLIT_COMPACT:
        # up to two accumulator/multiplier pairs per SIMD: a SIMD's share of
        # both netlists, or one accumulator's chain, whichever is longer
        G = ops["mul"] + ops["accum"]
        per_simd = -(-chain_waves // N_SIMD)
        clocks = max(taps * ops["accum"] * ISSUE_CLOCKS, taps * per_simd * G * SIMD_CLOCKS)
    else:
        G = ops["mac"]
        wgs_per_cu = -(-((P + 255) // 256) * ((d.M + 31) // 32) // N_CU)
        clocks = taps * G * max(ISSUE_CLOCKS, wgs_per_cu * SIMD_CLOCKS)
    lane_ops = P * d.M * taps / 32.0 * G
    return min(1.0, lane_ops / (clocks / CLOCK_HZ) / PEAK_LANE_OPS)


def pack_bench(reps):
    """Pack and unpack alone, on the element-wise workload's first operand
    (2^24 float32 values, (5,3)): one JSON line each, GB/s against 8 TB/s.
    Algorithmic bytes: 4 B per value read + the planes written (pack), the
    reverse for unpack."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    wE, wF = 5, 3
    a = torch.from_numpy(I.fma_operands(I.FMA_FORMATS.index((wE, wF)))[0].reshape(1, -1)).to(dev)
    n = a.numel()
    pa = hf.pack(a, (wE, wF))
    back = torch.empty_like(a)
    nbytes = n * 4 + pa.numel() * 4
    for name, fn in (("pack_kernel", lambda: hf.pack(a, (wE, wF), out=pa)),
                     ("unpack_kernel", lambda: hf.unpack(pa, 1, n, (wE, wF), kind="f32",
                                                         out=back))):
        ms = _time(fn, reps, stream)
        print(json.dumps({
            "workload": f"{name.split('_')[0]} 2^24 float32 values, ({wE},{wF}), "
                        f"{nbytes} algorithmic bytes", "kernel": name, "ms": ms,
            "roofline": {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9, "peak": 8000.0,
                         "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / HBM_PEAK}}), flush=True)


PROBE_KINDS = ["v_bitop3_b32 (8 bytes), sources in three VGPR banks, independent",
               "v_bitop3_b32, two sources in one VGPR bank, independent",
               "v_xor_b32 (VOP2, 4 bytes), sources in two banks, independent",
               "v_bitop3_b32, three banks, 1024 instructions per loop branch",
               "v_bitop3_b32, three banks, each reading the previous result",
               "v_bitop3_b32 and v_xor_b32 alternating, independent",
               "v_bitop3_b32, three banks, each reading the result two back",
               "v_bitop3_b32, three banks, each reading the result four back",
               "v_bitop3_b32, three banks, every instruction 8-byte aligned",
               "groups of one v_xor_b32 and seven v_bitop3_b32, every other group misaligned",
               "groups of v_xor_b32, seven v_bitop3_b32 and s_nop 0, all aligned"]


def issue_rate(iters):
    """The VALU issue-rate probe (csrc/issue_probe.hip): one JSON line per
    instruction stream and waves per CU (one workgroup per CU): how often one
    wave issues, how often one SIMD does, and the shader clock meanwhile. The
    single-wave interval is what the convolution's issue_ceiling rests on."""
    import ctypes
    from paper_2007_06563_amd import build as B
    L = ctypes.CDLL(B.PROBE_LIB)
    dbl = ctypes.POINTER(ctypes.c_double)
    L.hobflops_probe_issue.argtypes = [ctypes.c_int] * 4 + [dbl] * 3
    L.hobflops_probe_issue.restype = ctypes.c_int
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    runs = [(k, 1) for k in range(len(PROBE_KINDS))]
    runs += [(k, w) for k in (8, 1, 2, 4) for w in (2, 4, 8, 16)]
    for kind, waves in runs:
        a, b, c = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        rc = L.hobflops_probe_issue(cus, waves, kind, iters, ctypes.byref(a),
                                    ctypes.byref(b), ctypes.byref(c))
        if rc != 0:
            raise RuntimeError(f"issue probe failed: {rc}")
        print(json.dumps({
            "probe": "VALU issue rate", "stream": PROBE_KINDS[kind], "kind": kind,
            "waves_per_cu": waves, "waves_per_simd": -(-waves // 4),
            "clocks_per_instr_per_wave": round(a.value, 4),
            "clocks_per_instr_per_simd": round(b.value, 4),
            "shader_ghz": round(c.value, 4)}), flush=True)


def suite(reps, only=None):
    """One JSON line per further workload: the element-wise sweep and
    pack/unpack against HBM, the mantissa sweep and the 13-layer stack
    against the VALU peak. Inputs resident in HBM; kernels only. With `only`,
    just the workloads whose label contains that text (for profiling one)."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)

    def want(label):
        return only is None or only in label

    if want("device copy"):
        # what a plain device-to-device copy reaches on this GPU: the practical
        # HBM ceiling the HBM-bound kernels are compared with
        a = torch.empty(1 << 26, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        ms = _time(lambda: b.copy_(a), reps, stream)
        print(json.dumps({
            "workload": "device copy 256 MiB (reference for the HBM-bound kernels)",
            "kernel": "torch copy_", "ms": ms,
            "roofline": {"bound": "hbm", "achieved": 2 * a.numel() * 4 / (ms * 1e-3) / 1e9,
                         "peak": 8000.0, "unit": "GB/s",
                         "frac": 2 * a.numel() * 4 / (ms * 1e-3) / HBM_PEAK}}), flush=True)
        del a, b
    for idx, (wE, wF) in enumerate(I.FMA_FORMATS):
        if not want(f"element-wise a*b+c, 2^24 triples, ({wE},{wF}) -> ({wE},{wF + 1})"):
            continue
        a, b, c = (torch.from_numpy(t.reshape(1, -1)).to(dev) for t in I.fma_operands(idx))
        n = a.numel()
        f, fa = (wE, wF), (wE, wF + 1)
        pa, pb, pc = (hf.pack(t, f) for t in (a, b, c))
        r = hf.muladd(pa, pb, pc, n, f, fa)
        ms = _time(lambda: hf.muladd(pa, pb, pc, n, f, fa, out=r), reps, stream)
        nbytes = (3 * pa.numel() + r.numel()) * 4
        ms_pack = _time(lambda: hf.pack(a, f, out=pa), reps, stream)
        ms_unpack = _time(lambda: hf.unpack(r, 1, n, fa, kind="f32"), reps, stream)
        print(json.dumps({
            "workload": f"element-wise a*b+c, 2^24 triples, ({wE},{wF}) -> ({wE},{wF + 1})",
            "kernel": "muladd_kernel", "ms": ms, "gops": n / (ms * 1e-3) / 1e9,
            "roofline": {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9, "peak": 8000.0,
                         "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / HBM_PEAK},
            "pack_gbps": (n * 4 + pa.numel() * 4) / (ms_pack * 1e-3) / 1e9,
            "unpack_gbps": (r.numel() * 4 + n * 4) / (ms_unpack * 1e-3) / 1e9}), flush=True)
        del a, b, c, pa, pb, pc, r
    for si, s in enumerate(I.MANTISSA_SWEEP_SHAPES):
        for m in I.MANTISSA_SWEEP_WF:
            label = f"conv {s.N}x{s.H}x{s.W}x{s.C} -> {s.M} 3x3, (5,{m}) -> (5,{m + 1})"
            if not want(label):
                continue
            ifm, w = I.mantissa_sweep_inputs(si, m)
            d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, m),
                             (5, m + 1), (5, m + 1))
            pi = hf.pack(torch.from_numpy(ifm.reshape(-1, s.C)).to(dev), (5, m))
            pw = hf.pack(torch.from_numpy(w.reshape(-1, s.M)).to(dev), (5, m))
            o = hf.conv2d(pi, pw, d)
            ms = _time(lambda: hf.conv2d(pi, pw, d, out=o), reps, stream)
            algo, G = _conv_ops(d)
            lane_ops = s.macs / 32.0 * G
            print(json.dumps({
                "workload": label,
                "kernel": KERNEL_NAME[algo], "ms": ms,
                "gmacs": s.macs / (ms * 1e-3) / 1e9, "ops_per_mac_word": G,
                "roofline": {"bound": "alu", "achieved": lane_ops / (ms * 1e-3) / 1e12,
                             "peak": PEAK_LANE_OPS / 1e12, "unit": "T VALU-op/s",
                             "frac": lane_ops / (ms * 1e-3) / PEAK_LANE_OPS,
                             "issue_ceiling": issue_ceiling(d, algo)}}), flush=True)
    shapes = I.resnet_stack_shapes(16)
    fmts = I.resnet_stack_formats(len(shapes))
    stack_labels = [f"stack layer {li + 1}: {s.N}x{s.H}x{s.W}x{s.C} -> {s.M} {s.KH}x{s.KW} "
                    f"s{s.stride}, (5,{fmts[li][0]}) -> (5,{fmts[li][1]}) -> (5,{fmts[li][2]}) relu"
                    for li, s in enumerate(shapes)]
    stack_label = "13-layer stack, batch 16, 56x56x64 input, planes resident between layers"
    pool_labels = ["global average pooling, 13-layer stack output: 16x7x7x512, (5,4)",
                   "global average pooling, MobileNets interface: 16x7x7x1024, (5,4)"]
    if not any(want(x) for x in stack_labels + [stack_label] + pool_labels):
        return
    ifm0, _ = I.conv_inputs(I.RESNET_STACK, 0, shapes[0])
    x0 = hf.pack(torch.from_numpy(ifm0.reshape(-1, shapes[0].C)).to(dev), (5, fmts[0][0]))
    layers = []
    for li, (s, (wi, wa, wo)) in enumerate(zip(shapes, fmts)):
        _, w = I.conv_inputs(I.RESNET_STACK, li, s)
        d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (5, wi), (5, wa),
                         (5, wo), hf.ACT_RELU)
        pw = hf.pack(torch.from_numpy(w.reshape(-1, s.M)).to(dev), (5, wi))
        layers.append((s, d, pw))
    acts = [x0]
    for s, d, pw in layers:
        acts.append(hf.conv2d(acts[-1], pw, d))
    total_ms, total_macs, total_ops = 0.0, 0, 0.0
    for li, (s, d, pw) in enumerate(layers):
        algo, G = _conv_ops(d)
        total_macs += s.macs
        total_ops += s.macs / 32.0 * G
        if not want(stack_labels[li]):
            continue
        src, dst = acts[li], acts[li + 1]
        ms = _time(lambda: hf.conv2d(src, pw, d, out=dst), reps, stream)
        total_ms += ms
        print(json.dumps({
            "workload": stack_labels[li],
            "kernel": KERNEL_NAME[algo], "ms": ms,
            "gmacs": s.macs / (ms * 1e-3) / 1e9, "ops_per_mac_word": G,
            "roofline": {"bound": "alu", "achieved": s.macs / 32.0 * G / (ms * 1e-3) / 1e12,
                         "peak": PEAK_LANE_OPS / 1e12, "unit": "T VALU-op/s",
                         "frac": s.macs / 32.0 * G / (ms * 1e-3) / PEAK_LANE_OPS,
                         "issue_ceiling": issue_ceiling(d, algo)}}), flush=True)
    if not want(stack_label) and not any(want(x) for x in pool_labels):
        return

    def whole():
        for li, (s, d, pw) in enumerate(layers):
            hf.conv2d(acts[li], pw, d, out=acts[li + 1])
    if want(stack_label):
        ms = _time(whole, max(1, reps // 4), stream)
        print(json.dumps({
            "workload": stack_label,
            "ms": ms, "sum_of_layers_ms": total_ms, "gmacs": total_macs / (ms * 1e-3) / 1e9,
            "roofline": {"bound": "alu", "achieved": total_ops / (ms * 1e-3) / 1e12,
                         "peak": PEAK_LANE_OPS / 1e12, "unit": "T VALU-op/s",
                         "frac": total_ops / (ms * 1e-3) / PEAK_LANE_OPS}}), flush=True)
    # global average pooling in the packed format: the stack's last 7 x 7 x 512
    # map, and the MobileNets interface shape 7 x 7 x 1024, both batch 16
    s_last = shapes[-1]
    x1024 = hf.pack(torch.from_numpy(np.random.default_rng(5).normal(
        size=(16 * 49, 1024)).astype(np.float32)).to(dev), (5, 4))
    for label, src, C in ((pool_labels[0], acts[-1], s_last.M), (pool_labels[1], x1024, 1024)):
        if not want(label):
            continue
        N, H, W = 16, 7, 7
        f = (5, 4)
        o = hf.avgpool(src, N, H, W, C, f, f, f)
        ms = _time(lambda: hf.avgpool(src, N, H, W, C, f, f, f, out=o), reps, stream)
        ops = hf.avgpool_netlist_ops(f, f, f)
        words = N * ((C + 31) // 32)
        lane_ops = words * (H * W * ops["accum"] + ops["scale"])
        chain_us = H * W * ops["accum"] * ISSUE_CLOCKS / 2.3e3
        print(json.dumps({
            "workload": label,
            "kernel": "avgpool_kernel", "ms": ms, "g_adds": N * C * H * W / (ms * 1e-3) / 1e9,
            "chain_bound_us": chain_us, "lanes": words,
            "roofline": {"bound": "alu", "achieved": lane_ops / (ms * 1e-3) / 1e12,
                         "peak": PEAK_LANE_OPS / 1e12, "unit": "T VALU-op/s",
                         "frac": lane_ops / (ms * 1e-3) / PEAK_LANE_OPS}}), flush=True)


def sweep(reps):
    """The paper's type sweep (Table 3, Sec. 4): every generated MAC type,
    single and extended, rounding to nearest even and toward zero, on the
    MobileNets-shaped layer at batch 1 (the paper's shape) and batch 64; one
    JSON line each with the netlist gate counts (VALU instructions per 32-MAC
    word, the analogue of the paper's cell counts)."""
    from paper_2007_06563_amd import variants as V
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    names = {(4, 3): "HOBFLOPSIEEE8"}
    names.update({(5, m): f"HOBFLOPS{m + 6}" for m in range(2, 11)})
    for wE, wi, wa, wo, act, rnd in V.CONV_VARIANTS:
        if act or (wE, wi) not in names:
            continue
        ext = wa == 2 * wi + 1 and wa != wi + 1
        tname = names[(wE, wi)] + ("e" if ext else "")
        ops = hf.netlist_ops((wE, wi), (wE, wa), rnd)
        for batch in (1, 64):
            s = I.mobilenet_layer(batch)
            ifm, w = I.type_sweep_inputs(batch)
            d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, (wE, wi),
                             (wE, wa), (wE, wo), round=rnd)
            pi = hf.pack(torch.from_numpy(ifm.reshape(-1, s.C)).to(dev), (wE, wi))
            pw = hf.pack(torch.from_numpy(w.reshape(-1, s.M)).to(dev), (wE, wi))
            o = hf.conv2d(pi, pw, d)
            ms = _time(lambda: hf.conv2d(pi, pw, d, out=o), reps, stream)
            algo, G = _conv_ops(d)
            if G == 0:  # no split kernel for this type: the library ran the fused one
                algo, G = hf.ALGO_FUSED, ops["mac"]
            lane_ops = s.macs / 32.0 * G
            print(json.dumps({
                "type": tname, "in": [wE, wi], "acc": [wE, wa], "round": V.RND_NAME[rnd],
                "gates": {"mac": ops["mac"], "mul": ops["mul"], "accum": ops["accum"],
                          "muladd": ops["muladd"]},
                "workload": f"conv {s.N}x{s.H}x{s.W}x{s.C} -> {s.M} 3x3 s2 p1",
                "kernel": KERNEL_NAME[algo], "ms": ms,
                "gmacs": s.macs / (ms * 1e-3) / 1e9,
                "roofline": {"bound": "alu", "achieved": lane_ops / (ms * 1e-3) / 1e12,
                             "peak": PEAK_LANE_OPS / 1e12, "unit": "T VALU-op/s",
                             "frac": lane_ops / (ms * 1e-3) / PEAK_LANE_OPS,
                             "issue_ceiling": issue_ceiling(d, algo)}}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warmup-ms", type=float, default=400.0,
                    help="after the W warmup steps, keep running untimed steps until this "
                         "much time has passed, so that the GPU clock has ramped up")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB "
                         "(steps times): the reference for scaling HBM byte counters")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the one-line benchmark: the paper's MAC type sweep on the "
                         "MobileNets-shaped layer, one JSON line per type, rounding and batch")
    ap.add_argument("--pack", action="store_true",
                    help="instead of the one-line benchmark: pack and unpack alone on 2^24 "
                         "values, one JSON line each (for the HBM counters)")
    ap.add_argument("--suite", action="store_true",
                    help="instead of the one-line benchmark: one JSON line per further workload "
                         "(element-wise sweep, mantissa sweep, 13-layer stack)")
    ap.add_argument("--only", default=None,
                    help="with --suite: only the workloads whose label contains this text")
    ap.add_argument("--issue-rate", action="store_true",
                    help="instead of the one-line benchmark: the VALU issue-rate probe, one JSON "
                         "line per waves-per-CU and bank pattern")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the layer shards "
              "by batch with no exchange, so a multi-GPU figure is the single-GPU one times N "
              "minus launch skew; no multi-GPU path is built.", file=sys.stderr)
        sys.exit(2)
    torch.cuda.init()
    dev = torch.device("cuda:0")
    if args.suite:
        suite(args.steps, args.only)
        return
    if args.issue_rate:
        issue_rate(400)
        return
    if args.pack:
        pack_bench(args.steps)
        return
    if args.sweep:
        sweep(args.steps)
        return
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(args.steps):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes_each_way": n * 4, "launches": args.steps}))
        return
    s = I.RESNET_CONV_SHAPE
    ifm, w = I.resnet_conv_inputs()
    P = s.N * s.OH * s.OW
    # the library's automatic choice of kernel shape (for this layer: split
    # multiply/accumulate waves, its accumulator waves leaving each SIMD at
    # most one)
    algo = hf.conv2d_algo(hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad,
                                       IN_FMT, ACC_FMT, OUT_FMT, hf.ACT_NONE, hf.ALGO_AUTO))
    # the last (here: only) layer writes float32 directly: the unpack is fused
    # into the convolution's epilogue
    d = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, IN_FMT, ACC_FMT,
                     OUT_FMT, hf.ACT_NONE, algo, ofm_kind=hf.OFM_F32)
    x_ifm = torch.from_numpy(ifm.reshape(s.N * s.H * s.W, s.C)).to(dev)
    x_w = torch.from_numpy(w.reshape(s.KH * s.KW * s.C, s.M)).to(dev)
    p_ifm = torch.empty(hf.plane_shape(s.N * s.H * s.W, s.C, IN_FMT), dtype=torch.int32, device=dev)
    p_w = torch.empty(hf.plane_shape(s.KH * s.KW * s.C, s.M, IN_FMT), dtype=torch.int32, device=dev)
    y = torch.empty((P, s.M), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        hf.pack_batch([(x_ifm, p_ifm), (x_w, p_w)], IN_FMT)  # one launch for both
        if ev:
            ev[1].record(stream)
        hf.conv2d(p_ifm, p_w, d, out=y)
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t_w = time.perf_counter()
    while (time.perf_counter() - t_w) * 1e3 < args.warmup_ms:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    # the timed region: K steps with nothing else on the stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    # the same K steps again, with HIP events on the launch stream around the
    # pack and the convolution of every step: the per-kernel durations. An
    # event record holds the stream for about 5 us, so these steps are not
    # the timed ones.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    pack_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    conv_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))

    macs = s.macs
    ops = hf.netlist_ops(IN_FMT, ACC_FMT)
    G = ops["mac"] if algo == hf.ALGO_FUSED else ops["mul"] + ops["accum"]
    lane_ops = macs / 32.0 * G          # 32 MACs per 32-bit word operation
    achieved = lane_ops / (conv_ms * 1e-3)
    ceiling = issue_ceiling(d, algo)
    pack_bytes = (s.N * s.H * s.W * s.C + s.KH * s.KW * s.C * s.M) * 4 + \
        (p_ifm.numel() + p_w.numel()) * 4
    d_codes = hf.conv_desc(s.N, s.H, s.W, s.C, s.M, s.KH, s.KW, s.stride, s.pad, IN_FMT, ACC_FMT,
                           OUT_FMT, hf.ACT_NONE, algo, ofm_kind=hf.OFM_CODE)
    codes = hf.conv2d(p_ifm, p_w, d_codes)  # the same outputs as codes, for the CPU check
    torch.cuda.synchronize()
    gpu_codes = codes.cpu().numpy().view(np.uint32).astype(np.uint64).reshape(s.N, s.OH, s.OW, s.M)

    res = {
        "metric": "custom-FP conv GMAC/s and % of peak VALU bitwise-op rate, 9-bit fmt",
        "value": macs / (ms_step * 1e-3) / 1e9,
        "unit": "GMAC/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "e5m3 in, e5m4 acc, bitsliced on u32 planes",
        "data": "synthetic (seeded): IFM |N(0,1)| half zeroed, weights N(0,0.05)",
        "config": {"workload": "MCMK conv 8x56x56x64 -> 64 kernels 3x3, stride 1, pad 1, "
                               "HOBFLOPS9 (5,3)->(5,4), order (ky,kx,c); step = pack float32 IFM "
                               "and weights (one launch) + conv writing float32 OFM (unpack "
                               "fused into the epilogue)",
                   "macs_per_step": macs, "batch": s.N},
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12,
                     "unit": "T VALU-op/s (32-bit bitwise, one op = 32 gates)",
                     "frac": achieved / PEAK_LANE_OPS, "traffic": TRAFFIC,
                     "kernel": {1: "conv2d_kernel", 2: "conv2d_split_kernel",
                                3: "conv2d_split_compact_kernel"}[algo],
                     "ops_per_mac_word": G,
                     "kernel_ms": conv_ms,
                     "issue_ceiling": ceiling},
        "pct_valu_peak": 100.0 * achieved / PEAK_LANE_OPS,
        "conv_gmacs": macs / (conv_ms * 1e-3) / 1e9,
        "pack_ms": pack_ms,
        "pack_gbps": pack_bytes / (pack_ms * 1e-3) / 1e9,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(ifm, w, s, gpu_codes, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
