"""Host-side checks of the build: the guard against register copies of
in-flight inline-assembly loads (paper_2609_10264_amd/build.py)."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location("mvk_build", os.path.join(ROOT, "paper_2609_10264_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


KERNEL = """_Z6kernelv:
\t;;#ASMSTART
\tglobal_load_dwordx4 v[2:5], v[2:3], off
\t;;#ASMEND
{between}
\ts_waitcnt vmcnt(0)
\tv_mov_b32_e32 v7, v3
\ts_endpgm
"""


def test_copy_of_inflight_asm_load_is_flagged():
    b = _build_module()
    bad = b.asm_load_hazards(KERNEL.format(between="\tv_accvgpr_write_b32 a84, v5"))
    assert bad == [("_Z6kernelv", "v_accvgpr_write_b32 a84, v5")]
    assert len(b.asm_load_hazards(KERNEL.format(between="\tv_mov_b32_e32 v9, v[2:3]"))) == 1


def test_uses_after_the_drain_and_unrelated_copies_pass():
    b = _build_module()
    # the copy after vmcnt(0) reads a landed register; v8 was never an asm destination
    assert b.asm_load_hazards(KERNEL.format(between="\tv_mov_b32_e32 v9, v8")) == []
    # a compiler-issued load (outside inline assembly) is tracked by the compiler itself
    plain = KERNEL.replace(";;#ASMSTART", "").replace(";;#ASMEND", "")
    assert b.asm_load_hazards(plain.format(between="\tv_mov_b32_e32 v9, v5")) == []


SEQ = """_Z6kernelv:
\t;;#ASMSTART
\tglobal_load_dwordx4 v[2:5], v[10:11], off
\t;;#ASMEND
\tglobal_load_dwordx4 v[20:23], v[12:13], off
{between}
\ts_waitcnt vmcnt(0)
\ts_endpgm
"""


def test_writes_spills_and_loads_into_inflight_registers_are_flagged():
    b = _build_module()
    for ins in ("\tv_add_u32_e32 v3, v7, v8",                    # reuses an in-flight register
                "\tv_lshl_add_u64 v[4:5], v[30:31], 0, s[0:1]",  # the address of a later load
                "\tscratch_store_dwordx4 off, v[2:5], off",      # a spill of the stale value
                "\tbuffer_store_dword v5, off, s[0:3], 0",
                "\tglobal_load_dword v2, v[14:15], off"):         # a compiler load into it
        assert b.asm_load_hazards(SEQ.format(between=ins)) == [("_Z6kernelv", ins.strip())], ins


def test_a_covering_partial_wait_frees_the_registers():
    b = _build_module()
    # vmcnt(1): every vector-memory op but the most recent one has completed,
    # so the asm load (issued before the compiler's load) has landed
    ok = "\ts_waitcnt vmcnt(1)\n\tv_add_u32_e32 v3, v7, v8\n\tv_mov_b32_e32 v9, v4"
    assert b.asm_load_hazards(SEQ.format(between=ok)) == []
    # vmcnt(2) does not cover it: both loads may still be in flight
    bad = "\ts_waitcnt vmcnt(2)\n\tv_add_u32_e32 v3, v7, v8"
    assert b.asm_load_hazards(SEQ.format(between=bad)) == [("_Z6kernelv", "v_add_u32_e32 v3, v7, v8")]
    # writes of registers no asm load targets are fine
    assert b.asm_load_hazards(SEQ.format(between="\tv_add_u32_e32 v21, v7, v8")) == []
