"""ctypes binding of the C oracle (test infrastructure only).

Codes are numpy uint64 arrays in the LSB-first layout F | E | s | exn (see
hobflops_oracle.h). All functions are element-wise over equally shaped arrays.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("N", "H", "W", "C", "M", "KH", "KW", "stride", "pad",
                 "wE", "wF_in", "wF_acc", "wF_out", "act", "round")]

RNE, RTZ = 0, 1  # rounding modes: nearest with ties to even, toward zero


def load(path):
    """Load an oracle shared library from path and declare its signatures."""
    L = ctypes.CDLL(path)
    u64p = ctypes.POINTER(ctypes.c_uint64)
    f32p = ctypes.POINTER(ctypes.c_float)
    i64p = ctypes.POINTER(ctypes.c_int64)
    sz, ci = ctypes.c_size_t, ctypes.c_int
    L.hfo_quantize_f32_array.argtypes = [f32p, sz, ci, ci, u64p]
    L.hfo_decode_f32_array.argtypes = [u64p, sz, ci, ci, f32p]
    L.hfo_mul_array.argtypes = [u64p, u64p, sz, ci, ci, ci, u64p]
    L.hfo_add_array.argtypes = [u64p, u64p, sz, ci, ci, u64p]
    L.hfo_convert_array.argtypes = [u64p, sz, ci, ci, ci, u64p]
    L.hfo_relu_array.argtypes = [u64p, sz, ci, ci, u64p]
    L.hfo_muladd_array.argtypes = [u64p, u64p, u64p, sz, ci, ci, ci, u64p]
    L.hfo_mul_rm_array.argtypes = [u64p, u64p, sz, ci, ci, ci, ci, u64p]
    L.hfo_add_rm_array.argtypes = [u64p, u64p, sz, ci, ci, ci, u64p]
    L.hfo_convert_rm_array.argtypes = [u64p, sz, ci, ci, ci, ci, u64p]
    L.hfo_muladd_rm_array.argtypes = [u64p, u64p, u64p, sz, ci, ci, ci, ci, u64p]
    L.hfo_conv2d.argtypes = [u64p, u64p, u64p, ctypes.POINTER(ConvDesc), ci]
    L.hfo_conv2d_points.argtypes = [u64p, u64p, i64p, sz, u64p, ctypes.POINTER(ConvDesc), ci]
    L.hfo_recip.argtypes = [ctypes.c_uint64, ci, ci]
    L.hfo_recip.restype = ctypes.c_uint64
    L.hfo_avgpool.argtypes = [u64p, u64p, ci, ci, ci, ci, ci, ci, ci, ci, ci]
    for name in ("hfo_quantize_f32_array", "hfo_decode_f32_array", "hfo_mul_array",
                 "hfo_add_array", "hfo_convert_array", "hfo_relu_array",
                 "hfo_muladd_array", "hfo_conv2d", "hfo_conv2d_points",
                 "hfo_mul_rm_array", "hfo_add_rm_array", "hfo_convert_rm_array",
                 "hfo_muladd_rm_array", "hfo_avgpool",
                 "hfo_default_threads"):
        getattr(L, name).restype = ctypes.c_int
    return L


def lib():
    """The oracle library, compiled first if it is missing or stale."""
    global _lib
    if _lib is None:
        _lib = load(_build.build(force=False))
    return _lib


def _u64(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def _p(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t))


def _check(rc):
    if rc != 0:
        raise ValueError("oracle rejected the arguments (format or shape out of range)")


def default_threads() -> int:
    return lib().hfo_default_threads()


def quantize_f32(x, wE, wF, L=None):
    x = np.ascontiguousarray(x, dtype=np.float32)
    r = np.empty(x.shape, np.uint64)
    _check((L or lib()).hfo_quantize_f32_array(_p(x, ctypes.c_float), x.size, wE, wF, _p(r, ctypes.c_uint64)))
    return r


def decode_f32(codes, wE, wF, L=None):
    c = _u64(codes)
    r = np.empty(c.shape, np.float32)
    _check((L or lib()).hfo_decode_f32_array(_p(c, ctypes.c_uint64), c.size, wE, wF, _p(r, ctypes.c_float)))
    return r


def mul(a, b, wE, wF_in, wF_out, L=None, rnd=RNE):
    a, b = np.broadcast_arrays(_u64(a), _u64(b))
    a, b = _u64(a), _u64(b)
    r = np.empty(a.shape, np.uint64)
    _check((L or lib()).hfo_mul_rm_array(_p(a, ctypes.c_uint64), _p(b, ctypes.c_uint64), a.size, wE,
                                         wF_in, wF_out, rnd, _p(r, ctypes.c_uint64)))
    return r


def add(a, b, wE, wF, L=None, rnd=RNE):
    a, b = np.broadcast_arrays(_u64(a), _u64(b))
    a, b = _u64(a), _u64(b)
    r = np.empty(a.shape, np.uint64)
    _check((L or lib()).hfo_add_rm_array(_p(a, ctypes.c_uint64), _p(b, ctypes.c_uint64), a.size, wE,
                                         wF, rnd, _p(r, ctypes.c_uint64)))
    return r


def convert(a, wE, wF_src, wF_dst, L=None, rnd=RNE):
    a = _u64(a)
    r = np.empty(a.shape, np.uint64)
    _check((L or lib()).hfo_convert_rm_array(_p(a, ctypes.c_uint64), a.size, wE, wF_src, wF_dst,
                                             rnd, _p(r, ctypes.c_uint64)))
    return r


def relu(a, wE, wF, L=None):
    a = _u64(a)
    r = np.empty(a.shape, np.uint64)
    _check((L or lib()).hfo_relu_array(_p(a, ctypes.c_uint64), a.size, wE, wF, _p(r, ctypes.c_uint64)))
    return r


def muladd(a, b, c, wE, wF_in, wF_acc, L=None, rnd=RNE):
    a, b, c = np.broadcast_arrays(_u64(a), _u64(b), _u64(c))
    a, b, c = _u64(a), _u64(b), _u64(c)
    r = np.empty(a.shape, np.uint64)
    _check((L or lib()).hfo_muladd_rm_array(_p(a, ctypes.c_uint64), _p(b, ctypes.c_uint64),
                                            _p(c, ctypes.c_uint64), a.size, wE, wF_in, wF_acc,
                                            rnd, _p(r, ctypes.c_uint64)))
    return r


def _desc(ifm_shape, w_shape, stride, pad, wE, wF_in, wF_acc, wF_out, act, rnd):
    N, H, W, C = ifm_shape
    KH, KW, C2, M = w_shape
    if C2 != C:
        raise ValueError("channel mismatch between IFM and weights")
    return ConvDesc(N, H, W, C, M, KH, KW, stride, pad, wE, wF_in, wF_acc, wF_out, int(act),
                    int(rnd))


def conv2d(ifm, w, stride, pad, wE, wF_in, wF_acc, wF_out, act=0, nthreads=0, L=None, rnd=RNE):
    """Full convolution: ifm [N,H,W,C] and w [KH,KW,C,M] codes -> [N,OH,OW,M] codes."""
    ifm, w = _u64(ifm), _u64(w)
    d = _desc(ifm.shape, w.shape, stride, pad, wE, wF_in, wF_acc, wF_out, act, rnd)
    OH = (d.H + 2 * pad - d.KH) // stride + 1
    OW = (d.W + 2 * pad - d.KW) // stride + 1
    r = np.empty((d.N, OH, OW, d.M), np.uint64)
    _check((L or lib()).hfo_conv2d(_p(ifm, ctypes.c_uint64), _p(w, ctypes.c_uint64),
                            _p(r, ctypes.c_uint64), ctypes.byref(d), nthreads))
    return r


def conv2d_points(ifm, w, pts, stride, pad, wE, wF_in, wF_acc, wF_out, act=0, nthreads=0,
                  L=None, rnd=RNE):
    """Convolution outputs at the (n, oy, ox, m) rows of pts only."""
    ifm, w = _u64(ifm), _u64(w)
    pts = np.ascontiguousarray(pts, dtype=np.int64).reshape(-1, 4)
    d = _desc(ifm.shape, w.shape, stride, pad, wE, wF_in, wF_acc, wF_out, act, rnd)
    r = np.empty(len(pts), np.uint64)
    _check((L or lib()).hfo_conv2d_points(_p(ifm, ctypes.c_uint64), _p(w, ctypes.c_uint64),
                                   _p(pts, ctypes.c_int64), len(pts), _p(r, ctypes.c_uint64),
                                   ctypes.byref(d), nthreads))
    return r


def recip(n, wE, wF, L=None):
    """The code of 1/n in (wE, wF), rounded to nearest even."""
    r = (L or lib()).hfo_recip(int(n), wE, wF)
    if r == 0xFFFFFFFFFFFFFFFF:
        raise ValueError("oracle rejected the arguments (format or n out of range)")
    return np.uint64(r)


def avgpool(x, wE, wF_in, wF_acc, wF_out, L=None, rnd=RNE):
    """Global average pooling: x [N,H,W,C] codes -> [N,C] codes (hfo_avgpool)."""
    x = _u64(x)
    N, H, W, C = x.shape
    r = np.empty((N, C), np.uint64)
    _check((L or lib()).hfo_avgpool(_p(x, ctypes.c_uint64), _p(r, ctypes.c_uint64), N, H, W, C,
                                    wE, wF_in, wF_acc, wF_out, int(rnd)))
    return r
