"""The prefill kernels' LDS-DMA transfers (``buffer_load_dwordx4 ... lds``) take their LDS
destination in M0, which inline asm sets without declaring it: the compiler reserves M0
and rejects it as a clobber.  That is safe only while the compiler itself never uses M0
in these kernels.  This test holds that contract on the built code object (our own
gfx950 build of ``csrc/prefill_bf16.hip``, disassembled with the ROCm LLVM tools):

* every instruction that names M0 is an ``s_mov_b32 m0, sN`` immediately followed by an
  LDS-DMA transfer, and every LDS-DMA transfer immediately follows one;
* no instruction that reads M0 implicitly (relative register moves, messages, GWS,
  add-tid LDS access, interpolation) appears.

A toolchain that starts using M0 in these kernels fails here, on the CPU, before any
kernel runs.
"""
import re

from _codeobj import disassemble

IMPLICIT_M0 = re.compile(r"\b(v_movrel\w*|s_movrel\w*|s_sendmsg\w*|ds_gws\w*|ds_\w*addtid\w*|v_interp\w*|"
                         r"s_ttracedata)\b")


def m0_violations(ins):
    """Instructions that break the contract above (empty when it holds)."""
    bad = []
    for i, t in enumerate(ins):
        if t.startswith("buffer_load") and t.endswith(" lds"):
            if i == 0 or not re.fullmatch(r"s_mov_b32 m0, s\d+", ins[i - 1]):
                bad.append(t)
        if re.search(r"\bm0\b", t):
            nxt = ins[i + 1] if i + 1 < len(ins) else ""
            if not (re.fullmatch(r"s_mov_b32 m0, s\d+", t) and nxt.startswith("buffer_load") and nxt.endswith(" lds")):
                bad.append(t)
        if IMPLICIT_M0.search(t):
            bad.append(t)
    return bad


def test_checker_flags_other_m0_uses():
    ok = ["s_mov_b32 m0, s4", "buffer_load_dwordx4 v1, s[4:7], 0 offen lds", "v_mfma_f32_16x16x32_bf16 v[0:3], v[4:7], v[8:11], v[0:3]"]
    assert m0_violations(ok) == []
    assert m0_violations(["s_mov_b32 m0, s4", "v_movrels_b32 v0, v1"])           # M0 set, then used for indexing
    assert m0_violations(["buffer_load_dwordx4 v1, s[4:7], 0 offen lds"])         # transfer without its M0
    assert m0_violations(["s_mov_b32 m0, -1", "ds_read_b32 v0, v1"])              # compiler-written M0
    assert m0_violations(["s_sendmsg sendmsg(MSG_DEALLOC_VGPRS)"])


def test_m0_only_feeds_lds_dma(tmp_path):
    ins = disassemble("prefill_bf16.hip", tmp_path)
    assert len(ins) > 1000
    assert any(t.startswith("buffer_load") and t.endswith(" lds") for t in ins), "no LDS-DMA transfer found"
    assert m0_violations(ins) == []
