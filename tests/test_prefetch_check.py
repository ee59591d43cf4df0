"""The build-time check of the fused kernel's explicit prefetches (register
discipline between an inline-assembly load and its explicit wait)."""
import pytest

from paper_2310_10211_amd import check_prefetch

HEAD = "_ZN4gevo8k_fused2ILi256ELi128EEEvNS_10Fused2ArgsE:\n"
TAIL = ".Lfunc_end0:\n"


def _fn(body: str) -> str:
    return HEAD + body + TAIL


CLEAN = _fn("""\
.LBB0_1:
\t;;#ASMSTART
\ts_waitcnt vmcnt(0)
\t;;#ASMEND
\tv_add_f32_e32 v20, v8, v9
\t;;#ASMSTART
\tglobal_load_dwordx4 v[8:11], v[2:3], off
\t;;#ASMEND
\tv_mul_f32_e32 v21, v12, v13
\ts_cbranch_scc1 .LBB0_1
\ts_endpgm
""")


def test_clean_function_passes():
    assert check_prefetch.check_assembly(CLEAN) == {HEAD[:-2]: 1}


def test_use_before_wait_on_fallthrough_is_caught():
    bad = CLEAN.replace("\ts_endpgm\n", "\tv_mov_b32_e32 v30, v9\n\ts_endpgm\n")
    with pytest.raises(RuntimeError, match="used before its wait"):
        check_prefetch.check_assembly(bad)


def test_use_through_a_branch_target_is_caught():
    bad = _fn("""\
\t;;#ASMSTART
\tglobal_load_dwordx4 v[8:11], v[2:3], off
\t;;#ASMEND
\ts_cbranch_execz .LBB0_3
\tv_mov_b32_e32 v1, 0
\t;;#ASMSTART
\ts_waitcnt vmcnt(0)
\t;;#ASMEND
\ts_endpgm
.LBB0_3:
\tv_mov_b32_e32 v10, 0
\ts_endpgm
""")
    with pytest.raises(RuntimeError, match="used before its wait"):
        check_prefetch.check_assembly(bad)


def test_missing_prefetch_is_reported():
    with pytest.raises(RuntimeError, match="no prefetch blocks"):
        check_prefetch.check_assembly(_fn("\ts_endpgm\n"))


def test_partial_wait_needs_enough_younger_memory_operations():
    # vmcnt(2) right after the prefetch leaves it in flight: the later use is a violation
    early = _fn("""\
\t;;#ASMSTART
\tglobal_load_dwordx4 v[8:11], v[2:3], off
\t;;#ASMEND
\t;;#ASMSTART
\ts_waitcnt vmcnt(2)
\t;;#ASMEND
\tv_mov_b32_e32 v1, v8
\ts_endpgm
""")
    with pytest.raises(RuntimeError, match="used before its wait"):
        check_prefetch.check_assembly(early)
    # two younger stores make vmcnt(2) cover the prefetch
    ok = early.replace("\t;;#ASMSTART\n\ts_waitcnt vmcnt(2)",
                       "\tglobal_store_dword v[4:5], v1, off\n\tglobal_store_dword v[4:5], v1, off offset:4\n"
                       "\t;;#ASMSTART\n\ts_waitcnt vmcnt(2)")
    assert check_prefetch.check_assembly(ok) == {HEAD[:-2]: 1}


# ------------------------------------------------- VALU -> SGPR -> memory hazard
def _hz(body: str) -> str:
    return _fn(body)


HAZARD = _hz("""\
\tv_readfirstlane_b32 s0, v130
\tv_readfirstlane_b32 s1, v131
\t;;#ASMSTART
\tglobal_load_dwordx4 v[8:11], v150, s[0:1]
\t;;#ASMEND
\t;;#ASMSTART
\ts_waitcnt vmcnt(0)
\t;;#ASMEND
\tv_add_f32_e32 v20, v8, v9
\ts_endpgm
""")


def test_sgpr_base_written_by_valu_just_before_an_asm_load_is_caught():
    with pytest.raises(RuntimeError, match="reads an SGPR fewer than 5 wait states"):
        check_prefetch.check_assembly(HAZARD)


def test_five_wait_states_clear_the_sgpr_hazard():
    ok = HAZARD.replace("\tv_readfirstlane_b32 s1, v131\n", "\tv_readfirstlane_b32 s1, v131\n\ts_nop 4\n")
    assert check_prefetch.check_assembly(ok) == {HEAD[:-2]: 1}


def test_scalar_alu_base_is_not_a_hazard():
    ok = HAZARD.replace("v_readfirstlane_b32 s0, v130", "s_add_u32 s0, s20, s2").replace(
        "v_readfirstlane_b32 s1, v131", "s_addc_u32 s1, s21, 0")
    assert check_prefetch.check_assembly(ok) == {HEAD[:-2]: 1}


def test_sgpr_hazard_through_a_loop_back_edge_is_caught():
    bad = _hz("""\
.LBB0_1:
\t;;#ASMSTART
\tglobal_load_dwordx4 v[8:11], v150, s[4:5]
\t;;#ASMEND
\t;;#ASMSTART
\ts_waitcnt vmcnt(0)
\t;;#ASMEND
\tv_add_f32_e32 v20, v8, v9
\tv_add_co_u32_e64 v40, s[4:5], v41, v42
\ts_cbranch_scc1 .LBB0_1
\ts_endpgm
""")
    with pytest.raises(RuntimeError, match="reads an SGPR"):
        check_prefetch.check_assembly(bad)
    hz = check_prefetch.sgpr_hazards(bad.split("\n"))
    assert len(hz) == 1 and "s[4:5]" in hz[0][2]


# ------------------------------------------ direct-to-LDS loads (scalar operands)
DMA_HEAD = "_ZN4gevo11k_pred_gemmILb0EEEvNS_12PredGemmArgsE:\n"
DMA = DMA_HEAD + """\
\ts_add_u32 s20, s6, 0x400
\t;;#ASMSTART
\ts_mov_b32 m0, s20
\ts_nop 0
\tglobal_load_lds_dwordx4 v12, s[8:9]
\t;;#ASMEND
\ts_endpgm
""" + TAIL


def test_direct_to_lds_load_with_scalar_operands_passes():
    assert check_prefetch.check_scalar_operands(DMA, "_ZN4gevo11k_pred_gemm") == {DMA_HEAD[:-2]: 1}


def test_lds_address_from_a_vector_register_is_caught():
    bad = DMA.replace("s_mov_b32 m0, s20", "s_mov_b32 m0, v140")
    with pytest.raises(RuntimeError, match="m0 is written from a vector register"):
        check_prefetch.check_scalar_operands(bad, "_ZN4gevo11k_pred_gemm")


def test_direct_to_lds_base_written_by_valu_just_before_is_caught():
    bad = DMA.replace("\ts_add_u32 s20, s6, 0x400\n", "\tv_readfirstlane_b32 s8, v3\n\tv_readfirstlane_b32 s9, v4\n")
    with pytest.raises(RuntimeError, match="reads an SGPR fewer than 5 wait states"):
        check_prefetch.check_scalar_operands(bad, "_ZN4gevo11k_pred_gemm")


def test_lds_address_from_vcc_lo_is_a_scalar_operand():
    ok = DMA.replace("\ts_add_u32 s20, s6, 0x400\n", "\ts_add_i32 vcc_lo, s6, 0x400\n").replace(
        "s_mov_b32 m0, s20", "s_mov_b32 m0, vcc_lo")
    assert check_prefetch.check_scalar_operands(ok, "_ZN4gevo11k_pred_gemm") == {DMA_HEAD[:-2]: 1}
    bad = ok.replace("s_mov_b32 m0, vcc_lo", "s_mov_b32 m0, v[12]")
    with pytest.raises(RuntimeError, match="m0 is written from a vector register"):
        check_prefetch.check_scalar_operands(bad, "_ZN4gevo11k_pred_gemm")
