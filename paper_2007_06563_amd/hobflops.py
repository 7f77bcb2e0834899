"""Python binding of libhobflops.so (ctypes).

Argument marshalling only: every step runs in the library's HIP kernels, on
torch's current stream; torch supplies device memory and streams. There is no
CPU fallback: a missing library or a host tensor raises.
Plane tensors are int32 (the bit patterns of PL32 words).
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhobflops.so")
_lib = None

SRC_F32, SRC_CODE_U32 = 0, 1
ACT_NONE, ACT_RELU = 0, 1
ROUND_NEAREST_EVEN, ROUND_TOWARD_ZERO, ORDER_KY_KX_C = 0, 1, 0
ALGO_AUTO, ALGO_FUSED, ALGO_SPLIT, ALGO_SPLIT_COMPACT = 0, 1, 2, 3
OFM_PLANES, OFM_F32, OFM_CODE = 0, 1, 2


class HobflopsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"hobflops status {status}: {msg}")
        self.status = status


class Fmt(ctypes.Structure):
    _fields_ = [("wE", ctypes.c_int), ("wF", ctypes.c_int)]

    def __repr__(self):
        return f"Fmt({self.wE}, {self.wF})"


class ConvDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("H", ctypes.c_int), ("W", ctypes.c_int),
                ("C", ctypes.c_int), ("M", ctypes.c_int), ("KH", ctypes.c_int),
                ("KW", ctypes.c_int), ("stride", ctypes.c_int), ("pad", ctypes.c_int),
                ("in_fmt", Fmt), ("acc_fmt", Fmt), ("out_fmt", Fmt),
                ("act", ctypes.c_int), ("round", ctypes.c_int), ("order", ctypes.c_int),
                ("algo", ctypes.c_int), ("ofm_kind", ctypes.c_int)]


class PackJob(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("kind", ctypes.c_int), ("rows", ctypes.c_int64),
                ("len", ctypes.c_int64), ("planes", ctypes.c_void_p)]


EXPORTS = ("hobflops_plane_words", "hobflops_pack", "hobflops_pack_batch", "hobflops_unpack",
           "hobflops_conv2d",
           "hobflops_conv2d_supported", "hobflops_conv2d_algo", "hobflops_muladd", "hobflops_muladd_supported",
           "hobflops_netlist_ops", "hobflops_avgpool", "hobflops_avgpool_supported",
           "hobflops_avgpool_netlist_ops", "hobflops_wait_failures", "hobflops_set_wait_limit",
           "hobflops_get_wait_limit", "hobflops_status_string")


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2007_06563_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.hobflops_plane_words.argtypes = [i64, i64, Fmt, ctypes.POINTER(i64)]
        L.hobflops_pack.argtypes = [vp, ci, i64, i64, Fmt, vp, vp]
        L.hobflops_pack_batch.argtypes = [ctypes.POINTER(PackJob), ci, Fmt, vp]
        L.hobflops_unpack.argtypes = [vp, i64, i64, Fmt, ci, vp, vp]
        L.hobflops_conv2d.argtypes = [vp, vp, vp, ctypes.POINTER(ConvDesc), vp]
        L.hobflops_conv2d_supported.argtypes = [ctypes.POINTER(ConvDesc)]
        L.hobflops_conv2d_algo.argtypes = [ctypes.POINTER(ConvDesc)]
        L.hobflops_muladd.argtypes = [vp, vp, vp, vp, i64, Fmt, Fmt, ci, vp]
        L.hobflops_muladd_supported.argtypes = [Fmt, Fmt, ci]
        L.hobflops_netlist_ops.argtypes = [Fmt, Fmt, ci] + [ctypes.POINTER(ci)] * 4
        L.hobflops_avgpool.argtypes = [vp, vp, ci, ci, ci, ci, Fmt, Fmt, Fmt, ci, vp]
        L.hobflops_avgpool_supported.argtypes = [Fmt, Fmt, Fmt, ci]
        L.hobflops_avgpool_netlist_ops.argtypes = [Fmt, Fmt, Fmt, ci] + [ctypes.POINTER(ci)] * 2
        L.hobflops_wait_failures.argtypes = [ctypes.POINTER(ctypes.c_uint32), ci]
        L.hobflops_set_wait_limit.argtypes = [ctypes.c_uint32]
        L.hobflops_get_wait_limit.argtypes = []
        L.hobflops_status_string.argtypes = [ci]
        L.hobflops_status_string.restype = ctypes.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = ci
        L.hobflops_get_wait_limit.restype = ctypes.c_uint32
        _lib = L
    return _lib


def fmt(f):
    return f if isinstance(f, Fmt) else Fmt(int(f[0]), int(f[1]))


def nb(f):
    f = fmt(f)
    return 3 + f.wE + f.wF


def _check(rc):
    if rc != 0:
        raise HobflopsError(rc, lib().hobflops_status_string(rc).decode())


def _ptr(t):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("hobflops operates on GPU tensors only")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _require(t, nbytes, name):
    """The library reads and writes through raw pointers: a tensor smaller than
    the call's extent is refused here, before any launch."""
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name}: {have} bytes, the call needs {nbytes}")


def _stream(t):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def plane_words(rows, length, f):
    w = ctypes.c_int64()
    _check(lib().hobflops_plane_words(rows, length, fmt(f), ctypes.byref(w)))
    return w.value


def plane_shape(rows, length, f):
    return (rows, (length + 31) // 32, nb(f))


def pack(src, f, rows=None, length=None, out=None):
    """float32 values or int32 codes [rows, length] (any shape whose last axis
    is the packed one) -> int32 planes [rows, ceil(length/32), NB]."""
    f = fmt(f)
    if length is None:
        length = src.shape[-1]
    if rows is None:
        rows = src.numel() // max(length, 1)
    if src.numel() != rows * length:
        raise ValueError("rows * length does not match the source size")
    if src.dtype == torch.float32:
        kind = SRC_F32
    elif src.dtype in (torch.int32, torch.uint32):
        kind = SRC_CODE_U32
    else:
        raise TypeError("pack takes float32 values or int32 codes")
    if out is None:
        out = torch.empty(plane_shape(rows, length, f), dtype=torch.int32, device=src.device)
    _require(out, 4 * plane_words(rows, length, f), "pack out")
    _check(lib().hobflops_pack(_ptr(src), kind, rows, length, f, _ptr(out), _stream(src)))
    return out


def pack_batch(items, f):
    """Several pack() calls of one format in one launch (per 8 tensors).
    items: sequence of (src, out) pairs with out None or a planes tensor, or
    bare src tensors; each src packed along its last axis, as pack() does.
    Returns the planes tensors in order. The launch goes to the current stream
    of the first source's device."""
    f = fmt(f)
    jobs, outs = [], []
    for it in items:
        src, out = it if isinstance(it, (tuple, list)) else (it, None)
        length = src.shape[-1] if src.dim() else 1
        rows = src.numel() // max(length, 1)
        if src.dtype == torch.float32:
            kind = SRC_F32
        elif src.dtype in (torch.int32, torch.uint32):
            kind = SRC_CODE_U32
        else:
            raise TypeError("pack takes float32 values or int32 codes")
        if out is None:
            out = torch.empty(plane_shape(rows, length, f), dtype=torch.int32, device=src.device)
        _require(out, 4 * plane_words(rows, length, f), "pack_batch out")
        jobs.append(PackJob(_ptr(src).value, kind, rows, length, _ptr(out).value))
        outs.append(out)
    if not jobs:
        return outs
    arr = (PackJob * len(jobs))(*jobs)
    first = items[0][0] if isinstance(items[0], (tuple, list)) else items[0]
    _check(lib().hobflops_pack_batch(arr, len(jobs), f, _stream(first)))
    return outs


def unpack(planes, rows, length, f, kind="f32", out=None):
    """int32 planes -> float32 values (kind 'f32') or int32 codes ('code'), [rows, length]."""
    f = fmt(f)
    k = SRC_F32 if kind == "f32" else SRC_CODE_U32
    if out is None:
        out = torch.empty((rows, length), dtype=torch.float32 if k == SRC_F32 else torch.int32,
                          device=planes.device)
    _require(planes, 4 * plane_words(rows, length, f), "unpack planes")
    _require(out, 4 * rows * length, "unpack out")
    _check(lib().hobflops_unpack(_ptr(planes), rows, length, f, k, _ptr(out), _stream(planes)))
    return out


def conv_desc(N, H, W, C, M, KH, KW, stride, pad, in_fmt, acc_fmt, out_fmt, act=ACT_NONE,
              algo=ALGO_AUTO, round=ROUND_NEAREST_EVEN, ofm_kind=OFM_PLANES):
    return ConvDesc(N, H, W, C, M, KH, KW, stride, pad, fmt(in_fmt), fmt(acc_fmt), fmt(out_fmt),
                    act, round, ORDER_KY_KX_C, algo, ofm_kind)


def conv_out_hw(d):
    return ((d.H + 2 * d.pad - d.KH) // d.stride + 1, (d.W + 2 * d.pad - d.KW) // d.stride + 1)


def conv2d(ifm, w, d, out=None):
    """ifm planes [N*H*W, ceil(C/32), NB_in], w planes [KH*KW*C, ceil(M/32), NB_in]
    -> ofm planes [N*OH*OW, ceil(M/32), NB_out]; with d.ofm_kind OFM_F32 / OFM_CODE,
    float32 values / int32 codes [N*OH*OW, M]."""
    OH, OW = conv_out_hw(d)
    if out is None:
        if d.ofm_kind == OFM_PLANES:
            out = torch.empty(plane_shape(d.N * OH * OW, d.M, d.out_fmt), dtype=torch.int32,
                              device=ifm.device)
        else:
            out = torch.empty((d.N * OH * OW, d.M), device=ifm.device,
                              dtype=torch.float32 if d.ofm_kind == OFM_F32 else torch.int32)
    if OH > 0 and OW > 0 and d.N > 0 and d.C > 0 and d.M > 0:
        _require(ifm, 4 * plane_words(d.N * d.H * d.W, d.C, d.in_fmt), "conv2d ifm")
        _require(w, 4 * plane_words(d.KH * d.KW * d.C, d.M, d.in_fmt), "conv2d w")
        _require(out, 4 * (plane_words(d.N * OH * OW, d.M, d.out_fmt) if d.ofm_kind == OFM_PLANES
                           else d.N * OH * OW * d.M), "conv2d out")
    _check(lib().hobflops_conv2d(_ptr(ifm), _ptr(w), _ptr(out), ctypes.byref(d), _stream(ifm)))
    return out


def conv2d_supported(d):
    return bool(lib().hobflops_conv2d_supported(ctypes.byref(d)))


def conv2d_algo(d):
    """The kernel shape (ALGO_FUSED, ALGO_SPLIT or ALGO_SPLIT_COMPACT) conv2d
    runs d in: d.algo, or what AUTO picks on the current device."""
    rc = lib().hobflops_conv2d_algo(ctypes.byref(d))
    if rc < 0:
        _check(rc)
    return rc


def muladd(a, b, c, n, in_fmt, acc_fmt, out=None, round=ROUND_NEAREST_EVEN):
    """Element-wise add(widen(c), mul(a, b)) on flat planes of n elements."""
    in_fmt, acc_fmt = fmt(in_fmt), fmt(acc_fmt)
    if out is None:
        out = torch.empty(plane_shape(1, n, acc_fmt), dtype=torch.int32, device=a.device)
    for t, name in ((a, "a"), (b, "b"), (c, "c")):
        _require(t, 4 * plane_words(1, n, in_fmt), f"muladd {name}")
    _require(out, 4 * plane_words(1, n, acc_fmt), "muladd out")
    _check(lib().hobflops_muladd(_ptr(a), _ptr(b), _ptr(c), _ptr(out), n, in_fmt, acc_fmt, round,
                                 _stream(a)))
    return out


def muladd_supported(in_fmt, acc_fmt, round=ROUND_NEAREST_EVEN):
    return bool(lib().hobflops_muladd_supported(fmt(in_fmt), fmt(acc_fmt), round))


def netlist_ops(in_fmt, acc_fmt, round=ROUND_NEAREST_EVEN):
    """dict of VALU ops per 32-lane word: conv 'mac' (fused step), 'mul' and 'accum'
    (the split kernel's two roles), element-wise 'muladd'; 0 where not generated."""
    v = [ctypes.c_int() for _ in range(4)]
    rc = lib().hobflops_netlist_ops(fmt(in_fmt), fmt(acc_fmt), round,
                                    *[ctypes.byref(x) for x in v])
    if rc != 0:
        raise HobflopsError(rc, lib().hobflops_status_string(rc).decode())
    return dict(zip(("mac", "mul", "accum", "muladd"), (x.value for x in v)))


def avgpool(planes, N, H, W, C, in_fmt, acc_fmt, out_fmt, out=None, round=ROUND_NEAREST_EVEN):
    """Global average pooling: planes [N*H*W, ceil(C/32), NB_in] -> [N, ceil(C/32), NB_out]."""
    in_fmt, acc_fmt, out_fmt = fmt(in_fmt), fmt(acc_fmt), fmt(out_fmt)
    if out is None:
        out = torch.empty(plane_shape(N, C, out_fmt), dtype=torch.int32, device=planes.device)
    if N > 0 and H > 0 and W > 0 and C > 0:
        _require(planes, 4 * plane_words(N * H * W, C, in_fmt), "avgpool planes")
        _require(out, 4 * plane_words(N, C, out_fmt), "avgpool out")
    _check(lib().hobflops_avgpool(_ptr(planes), _ptr(out), N, H, W, C, in_fmt, acc_fmt, out_fmt,
                                  round, _stream(planes)))
    return out


def avgpool_supported(in_fmt, acc_fmt, out_fmt, round=ROUND_NEAREST_EVEN):
    return bool(lib().hobflops_avgpool_supported(fmt(in_fmt), fmt(acc_fmt), fmt(out_fmt), round))


def avgpool_netlist_ops(in_fmt, acc_fmt, out_fmt, round=ROUND_NEAREST_EVEN):
    """dict of VALU ops per 32-lane word of the pooling netlists: 'accum', 'scale'."""
    v = [ctypes.c_int() for _ in range(2)]
    rc = lib().hobflops_avgpool_netlist_ops(fmt(in_fmt), fmt(acc_fmt), fmt(out_fmt), round,
                                            *[ctypes.byref(x) for x in v])
    if rc != 0:
        raise HobflopsError(rc, lib().hobflops_status_string(rc).decode())
    return dict(zip(("accum", "scale"), (x.value for x in v)))


def wait_failures(reset=True):
    """Give-ups of the split kernel's bounded waits on the current device since
    the last reset (synchronises the device); nonzero means some launch's
    results are invalid."""
    n = ctypes.c_uint32()
    _check(lib().hobflops_wait_failures(ctypes.byref(n), 1 if reset else 0))
    return n.value


def set_wait_limit(sleeps):
    """Bound, in sleeps, of every counter wait in later split-kernel launches
    (process-wide; 0 gives up at the first look that misses)."""
    _check(lib().hobflops_set_wait_limit(int(sleeps)))


def get_wait_limit():
    return int(lib().hobflops_get_wait_limit())
