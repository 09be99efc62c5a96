"""The inline asm in the kernels gets no compiler-inserted wait states: the
kernels' gfx950 assembly is checked for dependencies that end at an asm
operand too early (host only: hipcc cross-compiles), and the checker itself
is checked on planted cases."""
import pytest

from paper_2609_35140_amd import asm_hazards as H
from paper_2609_35140_amd import build as B


def _fn(body: str) -> str:
    return "_Zkernel:\n" + body + "\n\ts_endpgm\n"


ASM = "\t;;#ASMSTART\n{}\n\t;;#ASMEND"


def test_trans_result_read_by_asm_is_flagged():
    text = _fn("\tv_exp_f32_e32 v6, v6\n" + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
    found = H.scan(text)
    assert len(found) == 1 and "v_exp_f32_e32 v6" in found[0]


def test_one_wait_state_clears_the_trans_read():
    for between in ("\ts_nop 0\n", "\tv_mul_f32_e32 v2, v3, v4\n"):
        text = _fn("\tv_exp_f32_e32 v6, v6\n" + between + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
        assert H.scan(text) == []
    # the settled exp of the numerics header: the s_nop sits inside the asm
    text = _fn(ASM.format("\tv_exp_f32 v6, v5\n\ts_nop 0") + "\n" + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
    assert H.scan(text) == []


def test_trans_read_through_a_branch_is_flagged():
    text = _fn("\tv_exp_f32_e32 v6, v6\n\ts_cbranch_scc1 .LBB0_2\n\tv_mov_b32_e32 v6, 0\n.LBB0_2:\n"
               + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
    # the fall-through path rewrites v6; the branch path arrives one wait state
    # (the branch) after the exp, which is enough
    assert H.scan(text) == []
    # an MFMA result needs more: the branch path is flagged, the fall-through
    # path (with its s_nops) is not
    text = _fn("\tv_mfma_f32_16x16x32_bf16 v[4:7], v[8:11], v[12:15], v[4:7]\n\ts_cbranch_scc1 .LBB0_2\n"
               "\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n.LBB0_2:\n" + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
    found = H.scan(text)
    assert len(found) == 1 and "with 1 wait states" in found[0]
    # the same through an unconditional branch
    text = _fn("\tv_mfma_f32_16x16x32_bf16 v[4:7], v[8:11], v[12:15], v[4:7]\n\ts_branch .LBB0_2\n"
               ".LBB0_1:\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n.LBB0_2:\n" + ASM.format("\tv_fma_f32 v129, v6, v129, v2"))
    found = H.scan(text)
    assert len(found) == 1 and "with 1 wait states" in found[0]


def test_mfma_result_read_by_asm_is_flagged():
    text = _fn("\tv_mfma_f32_16x16x32_bf16 v[0:3], v[4:7], v[8:11], v[0:3]\n\tv_mov_b32_e32 v20, v21\n"
               + ASM.format("\tv_fma_f32 v30, v31, v30, v2"))
    found = H.scan(text)
    assert len(found) == 1 and "v_mfma" in found[0]
    text = _fn("\tv_mfma_f32_16x16x32_bf16 v[0:3], v[4:7], v[8:11], v[0:3]\n\ts_nop 7\n\ts_nop 7\n\ts_nop 2\n"
               + ASM.format("\tv_fma_f32 v30, v31, v30, v2"))
    assert H.scan(text) == []


def test_valu_written_sgpr_read_by_asm_load_is_flagged():
    text = _fn("\tv_readfirstlane_b32 s4, v1\n\ts_mov_b32 s5, 0\n"
               + ASM.format("\ts_mov_b32 m0, s8\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v2, s[4:5]"))
    found = H.scan(text)
    assert len(found) == 1 and "v_readfirstlane_b32 s4" in found[0]
    text = _fn("\tv_readfirstlane_b32 s4, v1\n\ts_nop 4\n"
               + ASM.format("\ts_mov_b32 m0, s8\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v2, s[4:5]"))
    assert H.scan(text) == []


def _have_hipcc() -> bool:
    try:
        B.hipcc()
        return True
    except RuntimeError:
        return False


@pytest.mark.skipif(not _have_hipcc(), reason="hipcc is required")
def test_kernels_have_no_inline_asm_hazards():
    results = H.check()
    assert set(results) == set(H.SOURCES)
    bad = {src: found for src, found in results.items() if found}
    assert not bad, bad
