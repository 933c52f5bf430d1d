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
