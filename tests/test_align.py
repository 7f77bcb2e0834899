"""The 8-byte instruction alignment pass over device assembly (gen/align.py),
checked on small hand-written gfx950 code through the assembler itself."""
import os
import subprocess

import pytest

from paper_2007_06563_amd.gen import align

MC = "/opt/rocm/llvm/bin/llvm-mc"
pytestmark = pytest.mark.skipif(not os.path.exists(MC), reason="llvm-mc not installed")

HEAD = """\t.amdgcn_target "amdgcn-amd-amdhsa--gfx950"
\t.section\t.text.k,"ax",@progbits
\t.globl\tk
\t.p2align\t8
\t.type\tk,@function
k:
"""
OP = "\tv_bitop3_b32 v1, v2, v3, v4 bitop3:0x96\n"


def run(body, tmp_path, **kw):
    text = HEAD + body + "\ts_endpgm\n"
    src = tmp_path / "k.s"
    src.write_text(text)
    sizes = align.encoding_sizes(str(src), MC)
    before = align.misaligned_8byte(sizes, text)
    new, stats = align.align_text(text, sizes, **kw)
    out = tmp_path / "k_aligned.s"
    out.write_text(new)
    sizes2 = align.encoding_sizes(str(out), MC)
    after = align.misaligned_8byte(sizes2, new)
    r = subprocess.run([MC, "-triple=amdgcn-amd-amdhsa", "-mcpu=gfx950", "-filetype=obj",
                        "-o", str(tmp_path / "k.o"), str(out)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return new, stats, before, after, sizes, sizes2


def test_four_byte_valu_is_reencoded(tmp_path):
    new, st, before, after, s1, s2 = run("\tv_xor_b32_e32 v0, v1, v2\n" + OP * 8, tmp_path)
    assert before == (8, 8) and after == (0, 9)  # the re-encoded xor is the ninth
    assert st["promoted"] == 1 and st["nops"] == 0
    assert "v_xor_b32_e64 v0, v1, v2" in new
    assert len(s2) == len(s1)  # same instructions, one of them longer


def test_run_without_valu_gets_a_nop_before_a_long_stretch(tmp_path):
    new, st, before, after, s1, s2 = run("\ts_waitcnt lgkmcnt(0)\n" + OP * 8, tmp_path)
    assert before == (8, 8) and after == (0, 8)
    assert st["nops"] == 1 and st["promoted"] == 0
    assert len(s2) == len(s1) + 1
    # the nop goes in front of the run, before the wait
    assert new.index("s_nop 0") < new.index("s_waitcnt")


def test_short_stretch_is_left(tmp_path):
    # two misaligned instructions, then a 4-byte instruction restores the
    # alignment by itself: a nop would cost more than it saves
    body = "\ts_waitcnt lgkmcnt(0)\n" + OP * 2 + "\tv_xor_b32_e32 v0, v1, v2\n" + OP * 4
    new, st, before, after, s1, s2 = run(body, tmp_path)
    assert before == (2, 6) and after == (2, 6)
    assert st == {"promoted": 0, "nops": 0, "left": 1, "skipped_sections": 0}
    assert new == HEAD + body + "\ts_endpgm\n"


def test_carry_ops_are_not_reencoded(tmp_path):
    body = "\tv_add_co_u32_e32 v0, vcc, v1, v2\n" + OP * 8
    new, st, before, after, s1, s2 = run(body, tmp_path)
    assert "v_add_co_u32_e32" in new and st["promoted"] == 0 and st["nops"] == 1
    assert after == (0, 8)
    assert not align.promotable("v_addc_co_u32_e32") and not align.promotable("v_cmpx_eq_u32_e32")
    assert align.promotable("v_cndmask_b32_e32") and align.promotable("v_mov_b32_e32")


def test_only_named_sections_change(tmp_path):
    body = "\tv_xor_b32_e32 v0, v1, v2\n" + OP * 8
    new, st, before, after, s1, s2 = run(body, tmp_path, only=("other_kernel",))
    assert new == HEAD + body + "\ts_endpgm\n" and before == after == (8, 8)


def test_alignment_directive_restarts_the_count(tmp_path):
    body = "\ts_waitcnt lgkmcnt(0)\n\t.p2align 3\n" + OP * 8
    new, st, before, after, s1, s2 = run(body, tmp_path)
    assert before == (0, 8) and st["nops"] == 0 and st["promoted"] == 0
