"""The C ABI on the host: the library loads, exports every function the header
declares, and rejects bad arguments before launching anything (CPU only --
none of these calls reaches the GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def hf():
    from paper_2007_06563_amd import hobflops
    if not os.path.exists(hobflops.LIB_PATH):
        from paper_2007_06563_amd import build
        build.build(verbose=False)
    hobflops.lib()
    return hobflops


def declared_functions():
    text = open(os.path.join(ROOT, "include", "hobflops.h")).read()
    return sorted(set(re.findall(r"\b(hobflops_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported(hf):
    names = declared_functions()
    assert len(names) >= 9
    L = hf.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(hf.EXPORTS)


def test_plane_words(hf):
    assert hf.plane_words(10, 64, (5, 3)) == 10 * 2 * 11
    assert hf.plane_words(3, 33, (5, 4)) == 3 * 2 * 12
    assert hf.plane_words(0, 5, (5, 3)) == 0
    with pytest.raises(hf.HobflopsError):
        hf.plane_words(-1, 5, (5, 3))
    with pytest.raises(hf.HobflopsError):
        hf.plane_words(1, 5, (9, 3))


FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: calls fail before launch
MISALIGNED = ctypes.c_void_p(0x10002)


def desc(hf, **kw):
    base = dict(N=1, H=8, W=8, C=4, M=8, KH=3, KW=3, stride=1, pad=1, in_fmt=(5, 3),
                acc_fmt=(5, 4), out_fmt=(5, 4), act=0)
    base.update(kw)
    return hf.conv_desc(**base)


@pytest.mark.parametrize("bad", [dict(N=0), dict(C=-1), dict(stride=0), dict(pad=-1),
                                 dict(KH=11), dict(acc_fmt=(4, 4)), dict(acc_fmt=(5, 2)),
                                 dict(in_fmt=(1, 3)), dict(out_fmt=(5, 30)), dict(act=7)])
def test_conv_rejects_bad_descriptors(hf, bad):
    d = desc(hf, **bad)
    assert hf.lib().hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(d), None) == -1
    assert not hf.conv2d_supported(d)


def test_conv_rejects_round_order_and_algo(hf):
    for field, value in (("round", 2), ("round", -1), ("order", 2), ("algo", 4), ("algo", -1),
                         ("ofm_kind", 3), ("ofm_kind", -1)):
        d = desc(hf)
        setattr(d, field, value)
        assert hf.lib().hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(d), None) == -1, field


def test_conv_null_misaligned_unsupported(hf):
    L = hf.lib()
    d = desc(hf)
    assert L.hobflops_conv2d(None, FAKE, FAKE, ctypes.byref(d), None) == -1
    assert L.hobflops_conv2d(FAKE, MISALIGNED, FAKE, ctypes.byref(d), None) == -3
    assert L.hobflops_conv2d(FAKE, FAKE, FAKE, None, None) == -1
    u = desc(hf, in_fmt=(5, 3), acc_fmt=(5, 9), out_fmt=(5, 9))
    assert not hf.conv2d_supported(u)
    assert L.hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(u), None) == -2
    assert hf.conv2d_supported(desc(hf))
    d = desc(hf)
    d.round = hf.ROUND_TOWARD_ZERO
    assert hf.conv2d_supported(d)


def test_split_kernel_availability(hf):
    """Every generated variant, the widest extended type included, has both
    kernel shapes; a format triple with no generated variant is refused for
    every kernel shape, before anything is launched."""
    wide = dict(in_fmt=(5, 10), acc_fmt=(5, 21), out_fmt=(5, 21))
    for algo in (hf.ALGO_FUSED, hf.ALGO_AUTO, hf.ALGO_SPLIT):
        assert hf.conv2d_supported(desc(hf, **wide, algo=algo))
    assert hf.netlist_ops((5, 10), (5, 21))["mul"] > 0
    missing = dict(in_fmt=(6, 3), acc_fmt=(6, 4), out_fmt=(6, 4))  # not generated
    for algo in (hf.ALGO_FUSED, hf.ALGO_AUTO, hf.ALGO_SPLIT, hf.ALGO_SPLIT_COMPACT):
        assert not hf.conv2d_supported(desc(hf, **missing, algo=algo))
        d = desc(hf, **missing, algo=algo)
        assert hf.lib().hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(d), None) == -2
    assert hf.conv2d_supported(desc(hf, algo=hf.ALGO_SPLIT))
    # the compact form (two workgroups per CU) exists where the netlists fit
    # 128 VGPRs: the bench format, not the widest extended type
    assert hf.conv2d_supported(desc(hf, algo=hf.ALGO_SPLIT_COMPACT))
    assert not hf.conv2d_supported(desc(hf, **wide, algo=hf.ALGO_SPLIT_COMPACT))
    d = desc(hf, **wide, algo=hf.ALGO_SPLIT_COMPACT)
    assert hf.lib().hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(d), None) == -2
    d = desc(hf, algo=4)  # no such kernel shape
    assert hf.lib().hobflops_conv2d(FAKE, FAKE, FAKE, ctypes.byref(d), None) == -1


def test_conv_algo_query(hf):
    """hobflops_conv2d_algo reports an explicit kernel shape as given (no
    device needed), refuses what conv2d would refuse, and resolves AUTO on a
    device (without one it reports the HIP error)."""
    for algo in (hf.ALGO_FUSED, hf.ALGO_SPLIT, hf.ALGO_SPLIT_COMPACT):
        assert hf.conv2d_algo(desc(hf, algo=algo)) == algo
    wide = dict(in_fmt=(5, 10), acc_fmt=(5, 21), out_fmt=(5, 21))
    assert hf.lib().hobflops_conv2d_algo(ctypes.byref(
        desc(hf, **wide, algo=hf.ALGO_SPLIT_COMPACT))) == -2
    assert hf.lib().hobflops_conv2d_algo(ctypes.byref(desc(hf, algo=4))) == -1
    assert hf.lib().hobflops_conv2d_algo(None) == -1
    rc = hf.lib().hobflops_conv2d_algo(ctypes.byref(desc(hf)))  # AUTO
    assert rc in (hf.ALGO_FUSED, hf.ALGO_SPLIT, hf.ALGO_SPLIT_COMPACT, -4)


def test_pack_unpack_argument_checks(hf):
    L = hf.lib()
    f = hf.Fmt(5, 3)
    assert L.hobflops_pack(FAKE, 0, 4, 40, hf.Fmt(5, 40), FAKE, None) == -1
    assert L.hobflops_pack(FAKE, 5, 4, 40, f, FAKE, None) == -1
    assert L.hobflops_pack(None, 0, 4, 40, f, FAKE, None) == -1
    assert L.hobflops_pack(MISALIGNED, 0, 4, 40, f, FAKE, None) == -3
    assert L.hobflops_pack(None, 0, 0, 40, f, None, None) == 0  # empty: nothing to do
    assert L.hobflops_unpack(FAKE, -1, 40, f, 0, FAKE, None) == -1
    assert L.hobflops_unpack(FAKE, 4, 40, f, 0, MISALIGNED, None) == -3


def test_pack_batch_argument_checks(hf):
    L = hf.lib()
    f = hf.Fmt(5, 3)
    J = hf.PackJob

    def batch(*jobs, fmt=f):
        arr = (J * max(len(jobs), 1))(*jobs)
        return L.hobflops_pack_batch(arr, len(jobs), fmt, None)

    good = J(FAKE, 0, 4, 40, FAKE)
    assert L.hobflops_pack_batch(None, 0, f, None) == 0     # nothing to do
    assert L.hobflops_pack_batch(None, 2, f, None) == -1    # jobs missing
    assert L.hobflops_pack_batch(None, -1, f, None) == -1
    assert batch(good, fmt=hf.Fmt(5, 40)) == -1             # NB > 32
    assert batch(J(None, 0, 0, 40, None), J(None, 1, 7, 0, None)) == 0  # empty jobs skipped
    # a bad job anywhere fails the call before anything is launched (the good
    # job's fake pointers would fault if it were)
    assert batch(good, J(FAKE, 5, 4, 40, FAKE)) == -1       # kind
    assert batch(good, J(FAKE, 0, -1, 40, FAKE)) == -1      # rows
    assert batch(good, J(None, 0, 4, 40, FAKE)) == -1       # null source
    assert batch(good, J(FAKE, 0, 4, 40, MISALIGNED)) == -3
    assert batch(good, J(FAKE, 0, 1 << 40, 1 << 40, FAKE)) == -1  # size overflow


def test_muladd_argument_checks(hf):
    L = hf.lib()
    a = hf.Fmt(5, 3)
    assert L.hobflops_muladd(FAKE, FAKE, FAKE, FAKE, -5, a, hf.Fmt(5, 4), 0, None) == -1
    assert L.hobflops_muladd(FAKE, FAKE, FAKE, FAKE, 64, a, hf.Fmt(4, 4), 0, None) == -1
    assert L.hobflops_muladd(FAKE, FAKE, FAKE, FAKE, 64, a, hf.Fmt(5, 4), 2, None) == -1
    assert L.hobflops_muladd(FAKE, FAKE, FAKE, FAKE, 64, a, hf.Fmt(5, 9), 0, None) == -2
    assert L.hobflops_muladd(FAKE, FAKE, None, FAKE, 64, a, hf.Fmt(5, 4), 0, None) == -1
    assert L.hobflops_muladd(FAKE, FAKE, FAKE, MISALIGNED, 64, a, hf.Fmt(5, 4), 0, None) == -3
    assert hf.muladd_supported((5, 3), (5, 4))
    assert hf.muladd_supported((5, 3), (5, 4), hf.ROUND_TOWARD_ZERO)
    assert not hf.muladd_supported((5, 3), (5, 9))


def test_netlist_ops_and_status_strings(hf):
    ops = hf.netlist_ops((5, 3), (5, 4))
    assert 50 < ops["mac"] < 1000 and 50 < ops["muladd"] < 1000
    assert 20 < ops["mul"] < ops["mac"] and 50 < ops["accum"] < ops["mac"]
    # toward zero drops the rounding logic: fewer instructions (paper Sec. 4)
    rtz = hf.netlist_ops((5, 3), (5, 4), hf.ROUND_TOWARD_ZERO)
    assert rtz["mac"] < ops["mac"] and rtz["accum"] < ops["accum"]
    assert rtz["muladd"] < ops["muladd"]
    with pytest.raises(hf.HobflopsError):
        hf.netlist_ops((5, 3), (5, 9))
    L = hf.lib()
    for s in (0, -1, -2, -3, -4, 12):
        assert L.hobflops_status_string(s)


def test_python_binding_refuses_host_tensors(hf):
    import torch
    with pytest.raises(TypeError):
        hf.pack(torch.zeros(4, 32), (5, 3))


def test_python_binding_refuses_short_buffers(hf):
    """The library works on raw pointers; the binding refuses tensors smaller
    than a call's extent before anything reaches the device (these tensors
    are on the host, so a call that got past the check would fail with
    TypeError instead)."""
    import torch
    i32 = torch.int32
    with pytest.raises(ValueError, match="pack out"):
        hf.pack(torch.zeros(4, 40), (5, 3), out=torch.zeros(4 * 2 * 11 - 1, dtype=i32))
    with pytest.raises(ValueError, match="pack_batch out"):
        hf.pack_batch([(torch.zeros(4, 40), torch.zeros(5, dtype=i32))], (5, 3))
    with pytest.raises(ValueError, match="unpack planes"):
        hf.unpack(torch.zeros(4 * 2 * 11 - 1, dtype=i32), 4, 40, (5, 3))
    with pytest.raises(ValueError, match="unpack out"):
        hf.unpack(torch.zeros(4 * 2 * 11, dtype=i32), 4, 40, (5, 3),
                  out=torch.zeros(4 * 40 - 1))
    d = hf.conv_desc(1, 4, 4, 40, 8, 3, 3, 1, 1, (5, 3), (5, 4), (5, 4))
    ifm_words, w_words = 16 * 2 * 11, 9 * 40 * 1 * 11
    with pytest.raises(ValueError, match="conv2d ifm"):
        hf.conv2d(torch.zeros(ifm_words - 1, dtype=i32), torch.zeros(w_words, dtype=i32), d)
    with pytest.raises(ValueError, match="conv2d w"):
        hf.conv2d(torch.zeros(ifm_words, dtype=i32), torch.zeros(w_words - 1, dtype=i32), d)
    with pytest.raises(ValueError, match="conv2d out"):
        hf.conv2d(torch.zeros(ifm_words, dtype=i32), torch.zeros(w_words, dtype=i32), d,
                  out=torch.zeros(16 * 12 - 1, dtype=i32))
    with pytest.raises(ValueError, match="muladd b"):
        hf.muladd(torch.zeros(11, dtype=i32), torch.zeros(10, dtype=i32),
                  torch.zeros(11, dtype=i32), 32, (5, 3), (5, 4))
    with pytest.raises(ValueError, match="avgpool planes"):
        hf.avgpool(torch.zeros(10, dtype=i32), 1, 2, 2, 32, (5, 4), (5, 4), (5, 4))


def test_avgpool_argument_checks(hf):
    L = hf.lib()
    f54, f55, f44 = hf.fmt((5, 4)), hf.fmt((5, 5)), hf.fmt((4, 4))
    ok = (FAKE, FAKE, 2, 7, 7, 64, f54, f54, f54, 0, None)
    # shapes, formats and rounding mode are checked before anything else
    for i, bad in ((2, 0), (3, 0), (4, -1), (5, 0), (9, 2)):
        args = list(ok)
        args[i] = bad
        assert L.hobflops_avgpool(*args) == -1, (i, bad)
    assert L.hobflops_avgpool(FAKE, FAKE, 1, 1 << 16, 1 << 16, 8, f54, f54, f54, 0, None) == -1
    assert L.hobflops_avgpool(FAKE, FAKE, 1, 2, 2, 8, f54, f44, f54, 0, None) == -1   # wE differs
    assert L.hobflops_avgpool(FAKE, FAKE, 1, 2, 2, 8, f55, f54, f54, 0, None) == -1   # acc narrower
    assert L.hobflops_avgpool(FAKE, FAKE, 1, 2, 2, 8, f54, f55, f55, 0, None) == -2   # not generated
    assert L.hobflops_avgpool(None, FAKE, 1, 2, 2, 8, f54, f54, f54, 0, None) == -1
    assert L.hobflops_avgpool(FAKE, MISALIGNED, 1, 2, 2, 8, f54, f54, f54, 0, None) == -3
    assert hf.avgpool_supported((5, 4), (5, 4), (5, 4))
    assert hf.avgpool_supported((5, 4), (5, 5), (5, 4), round=hf.ROUND_TOWARD_ZERO)
    assert not hf.avgpool_supported((5, 4), (5, 5), (5, 5))
    ops = hf.avgpool_netlist_ops((5, 4), (5, 4), (5, 4))
    assert ops["accum"] == hf.netlist_ops((5, 3), (5, 4))["accum"] and ops["scale"] > 0


def test_wait_limit_and_failure_query_arguments(hf):
    """The split kernel's wait bound is a process-wide setting read at launch;
    the give-up query refuses a NULL output before touching the device."""
    L = hf.lib()
    default = hf.get_wait_limit()
    assert default == 1 << 20
    try:
        hf.set_wait_limit(0)
        assert hf.get_wait_limit() == 0
        hf.set_wait_limit(12345)
        assert L.hobflops_get_wait_limit() == 12345
    finally:
        hf.set_wait_limit(default)
    assert L.hobflops_wait_failures(None, 0) == -1
