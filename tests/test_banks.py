"""The VGPR bank pass over device assembly (gen/banks.py), checked on small
hand-written gfx950 functions: fewer bank clashes, the same values read by
every instruction, nothing renamed across blocks, and the assembler accepts
the result."""
import os
import subprocess

import pytest

from paper_2007_06563_amd.gen import banks

MC = "/opt/rocm/llvm/bin/llvm-mc"

HEAD = """\t.amdgcn_target "amdgcn-amd-amdhsa--gfx950"
\t.section\t.text.kern,"ax",@progbits
\t.globl\tkern
\t.p2align\t8
\t.type\tkern,@function
kern:
"""


def wrap(body):
    return HEAD + body + "\ts_endpgm\n"


def assemble(text, tmp_path):
    if not os.path.exists(MC):
        pytest.skip("llvm-mc not installed")
    src = tmp_path / "k.s"
    src.write_text(text)
    r = subprocess.run([MC, "-triple=amdgcn-amd-amdhsa", "-mcpu=gfx950", "-filetype=obj",
                        "-o", str(tmp_path / "k.o"), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


# v0..v5 and v12 are memory operands (pinned); v9's first value and v10 are
# temporaries living inside the block: v9 meets v1 (bank 1) and v10 meets v2
# (bank 2) in the instructions that read them.
BODY = """\tglobal_load_dwordx4 v[0:3], v[4:5], off
\ts_waitcnt vmcnt(0)
\tv_bitop3_b32 v9, v0, v2, v3 bitop3:0x96
\tv_bitop3_b32 v10, v9, v1, v3 bitop3:0x80
\tv_bitop3_b32 v9, v10, v0, v2 bitop3:0xe8
\tv_mov_b32_e32 v12, v9
\tglobal_store_dword v[4:5], v12, off
"""


def test_clash_is_removed_and_values_kept(tmp_path):
    text = wrap(BODY)
    assert banks.count_conflicts(text) == 2
    new, st = banks.rename_text(text)
    assert st["blocks"] == 1 and (st["conflicts_before"], st["conflicts_after"]) == (2, 0)
    assert banks.count_conflicts(new) == 0
    assemble(new, tmp_path)
    lines = new.split("\n")
    # memory instructions and their registers are untouched
    assert "\tglobal_load_dwordx4 v[0:3], v[4:5], off" in lines
    assert "\tglobal_store_dword v[4:5], v12, off" in lines
    ops = [l.split(None, 1)[1].split(" bitop3")[0].split(", ")
           for l in lines if l.startswith("\tv_bitop3_b32")]
    a, b, c = ops
    # each reader reads the register its producer now writes
    assert b[1] == a[0] and c[1] == b[0]
    assert a[1:] == ["v0", "v2", "v3"] and b[2:] == ["v1", "v3"] and c[2:] == ["v0", "v2"]
    # the second value of v9 feeds the copy; v_mov reads what c writes
    mov = [l for l in lines if l.startswith("\tv_mov_b32")][0]
    assert mov.split(", ")[1] == c[0]


def test_value_live_into_another_block_is_not_renamed():
    # v8's first value is read after a branch: it is live out of its block
    body = """\tglobal_load_dwordx4 v[0:3], v[4:5], off
\ts_waitcnt vmcnt(0)
\tv_bitop3_b32 v8, v0, v1, v2 bitop3:0x96
\ts_cbranch_scc1 .LBB0_2
.LBB0_1:
\tv_bitop3_b32 v12, v8, v4, v3 bitop3:0x80
\tglobal_store_dword v[4:5], v12, off
.LBB0_2:
"""
    new, st = banks.rename_text(wrap(body))
    assert st["blocks"] == 0 and new == wrap(body)


def test_block_writing_exec_is_left_alone():
    body = BODY.replace("\ts_waitcnt vmcnt(0)\n",
                        "\ts_waitcnt vmcnt(0)\n\ts_and_saveexec_b64 s[0:1], vcc\n")
    new, st = banks.rename_text(wrap(body))
    assert st["blocks"] == 0 and new == wrap(body)


def test_register_indexing_leaves_the_function_alone():
    body = BODY + "\tv_movrels_b32_e32 v9, v10\n"
    new, st = banks.rename_text(wrap(body))
    assert st["skipped"] == 1 and new == wrap(body)


def test_only_named_functions_change():
    new, st = banks.rename_text(wrap(BODY), only=("other",))
    assert st["functions"] == 0 and new == wrap(BODY)
