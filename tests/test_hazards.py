"""The wait-state check of the device assembly: planted hazards in small
hand-written listings are found, legal spacing is not reported, and the
library's own device code (compiled here for gfx950) is clean."""
import os
import shutil
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2606_01502_amd import build as B
from paper_2606_01502_amd import hazards as Z


def _fn(body):
    return "_Zkernel:\n" + body + "\n\ts_endpgm\n.Lfunc_end0:\n"


def _asm(*lines):
    return "\t;;#ASMSTART\n" + "\n".join("\t" + x for x in lines) + "\n\t;;#ASMEND\n"


MFMA = "v_mfma_f32_16x16x32_bf16 v[4:7], v[8:11], v[12:15], v[4:7]"


def test_valu_copy_right_before_asm_product():
    # the pattern found in the fp8 kernel: a compiler copy into the
    # accumulator, then the product that reads it as SrcC
    text = _fn("\tv_mov_b32_e32 v6, v40\n" + _asm(MFMA))
    bad = Z.check(text)
    assert len(bad) == 1 and "needs 2 wait states, has 0" in bad[0]
    text = _fn("\tv_mov_b32_e32 v6, v40\n\tv_mov_b32_e32 v41, v40\n" + _asm(MFMA))
    assert "has 1" in Z.check(text)[0]
    # operands A and B count too
    assert Z.check(_fn("\tv_cvt_f32_f16_e32 v9, v40\n" + _asm(MFMA)))
    assert Z.check(_fn("\tv_add_u32_e32 v14, v40, v41\n" + _asm(MFMA)))


def test_swaps_write_both_operands():
    # the row-swap permutes (and v_swap) also write their second operand
    for op in ("v_permlane16_swap_b32_e32", "v_permlane32_swap_b32_e32", "v_swap_b32"):
        bad = Z.check(_fn(f"\t{op} v40, v6\n" + _asm(MFMA)))
        assert bad and "has 0" in bad[0], op
    assert Z.check(_fn("\tv_permlane16_swap_b32_e32 v40, v41\n" + _asm(MFMA))) == []


def test_enough_wait_states_pass():
    assert Z.check(_fn("\tv_mov_b32_e32 v6, v40\n" + _asm("s_nop 1", MFMA))) == []
    assert Z.check(_fn("\tv_mov_b32_e32 v6, v40\n\ts_nop 0\n\tv_mov_b32_e32 v41, v40\n" +
                       _asm(MFMA))) == []
    # unrelated registers
    assert Z.check(_fn("\tv_mov_b32_e32 v16, v40\n" + _asm(MFMA))) == []


def test_result_read_too_early():
    use = "\tv_max_f32_e32 v20, v5, v21\n"
    bad = Z.check(_fn(_asm(MFMA) + use))
    assert len(bad) == 1 and "needs 11" in bad[0]
    assert Z.check(_fn(_asm(MFMA, "s_nop 7", "s_nop 2") + use)) == []
    # a store of the result, and a write over it, count as well
    assert Z.check(_fn(_asm(MFMA) + "\tglobal_store_dwordx4 v[30:31], v[4:7], off\n"))
    assert Z.check(_fn(_asm(MFMA) + "\tv_mov_b32_e32 v7, 0\n"))
    # 32x32 shapes take longer
    big = "v_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], v[20:23], v[0:15]"
    bad = Z.check(_fn(_asm(big, "s_nop 7", "s_nop 2") + "\tv_mov_b32_e32 v30, v3\n"))
    assert bad and "needs 19" in bad[0]


def test_accumulation_chain_and_compiler_pairs():
    # back-to-back accumulation into the same registers is interlocked
    assert Z.check(_fn(_asm(MFMA, MFMA))) == []
    # a product reading the previous result as an A operand is not
    chained = "v_mfma_f32_16x16x32_bf16 v[20:23], v[4:7], v[12:15], 0"
    assert Z.check(_fn(_asm(MFMA, chained)))
    # neither instruction from inline asm: the compiler's own business
    assert Z.check(_fn("\tv_mov_b32_e32 v6, v40\n\t" + MFMA + "\n")) == []


def test_paths_through_branches():
    # the read sits at the loop head; the product ends the loop body
    loop = (".LBB0_1:\n\tv_max_f32_e32 v20, v5, v21\n\ts_nop 7\n" + _asm(MFMA) +
            "\ts_cbranch_scc1 .LBB0_1\n")
    bad = Z.check(_fn(loop))
    assert bad and "has 1" in bad[0]
    # an unconditional branch away: no fall-through into the next block
    text = _fn(_asm(MFMA) + "\ts_branch .LBB0_2\n.LBB0_3:\n\tv_max_f32_e32 v20, v5, v21\n"
               ".LBB0_2:\n\ts_nop 7\n\ts_nop 7\n\ts_cbranch_scc1 .LBB0_3\n")
    assert Z.check(text) == []


def test_library_device_code_is_clean(tmp_path):
    """Every kernel of the library, compiled here for gfx950."""
    if shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not available")
    old = B.BUILD_DIR
    B.BUILD_DIR = str(tmp_path)
    try:
        with ThreadPoolExecutor(max_workers=4) as ex:
            asms = list(ex.map(B._device_asm, B.sources()))
    finally:
        B.BUILD_DIR = old
    texts = [open(a).read() for a in asms]
    assert sum(t.count("v_mfma") for t in texts) > 100  # the products are there
    B.check_hazards(asms)
