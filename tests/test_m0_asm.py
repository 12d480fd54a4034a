"""The buffer->LDS loads of the large-tile products set M0 in inline assembly,
which the compiler cannot take into account (it ignores M0 in a clobber
list).  That is safe only while no compiler-generated instruction writes or
reads M0 in the same code object.  This test compiles that translation unit
for gfx950 to AMD assembly, with the library's flags, and checks:

* every instruction that names m0 is the assembly block's own
  `s_mov_b32 m0, sN`, followed by `s_nop 0` and its four
  `buffer_load_dwordx4 ... lds`;
* every buffer->LDS load sits in such a block;
* nothing else that reads M0 implicitly (relative moves, messages, GWS,
  append/consume, interpolation, GPR index mode, addtid LDS access, global
  loads to LDS) appears anywhere.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2608_01528_amd import build as B

SRC = os.path.join(B.CSRC, "gs_gemm256.hip")
IMPLICIT_M0 = re.compile(r"^(s_movrel|v_movrel|s_sendmsg|ds_gws|ds_append|ds_consume|v_interp|s_set_gpr_idx"
                         r"|ds_read_addtid|ds_write_addtid|global_load_lds|global_load_lds_)")
INSTR = re.compile(r"^\s+([a-z_][a-z0-9_]*)(\s.*)?$")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    hipcc = B.HIPCC
    if not (os.path.exists(hipcc) or shutil.which(hipcc)):
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "gs_gemm256.s")
    cmd = [hipcc] + B.FLAGS + ["--cuda-device-only", "-S", "-o", out, SRC]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


def instructions(text):
    """(function, mnemonic, operands) for every instruction line, comments
    stripped; the function is the last label declared @function."""
    funcs = set(re.findall(r"\.type\s+([^,\s]+),@function", text))
    cur = None
    for line in text.splitlines():
        line = line.split(";")[0].rstrip()
        m = re.match(r"^([^\s:]+):$", line)
        if m and m.group(1) in funcs:
            cur = m.group(1)
            continue
        m = INSTR.match(line)
        if m and not line.lstrip().startswith("."):
            yield cur, m.group(1), (m.group(2) or "").strip()


def test_m0_written_only_by_the_dma_blocks(asm):
    ins = list(instructions(asm))
    blocks = 0
    dma_funcs = set()
    in_block = 0                    # buffer->LDS loads still expected in the current block
    for i, (fn, op, args) in enumerate(ins):
        if re.search(r"\bm0\b", args):
            assert op == "s_mov_b32" and re.fullmatch(r"m0,\s*s\d+", args), (fn, op, args)
            assert in_block == 0, (fn, "M0 rewritten inside a block")
            assert ins[i + 1][1:] == ("s_nop", "0"), (fn, ins[i + 1])
            blocks += 1
            in_block = 4
            dma_funcs.add(fn)
            continue
        if op.startswith("buffer_load") and re.search(r"\blds\b", args):
            assert in_block > 0, (fn, op, args, "buffer->LDS load outside a block")
            assert op == "buffer_load_dwordx4"
            in_block -= 1
            continue
        if op == "s_nop" and in_block == 4:
            continue
        assert in_block == 0, (fn, op, args, "instruction inside a block")
        assert not IMPLICIT_M0.match(op), (fn, op, args)
    assert in_block == 0
    # the products do use the loads (the test is not vacuous)
    assert blocks > 0
    assert any("gemm256_store_kernel" in f for f in dma_funcs)
    assert any("scores256_kernel" in f for f in dma_funcs)
