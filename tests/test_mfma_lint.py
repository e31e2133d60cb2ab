"""The build-time MFMA check on small hand-written assembly fragments."""
from paper_1912_03203_amd import mfma_lint

HEAD = "_ZN7dynconv1kEv:\n"


def test_early_read_is_reported():
    asm = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	v_add_f32_e32 v12, v1, v13
"""
    found = mfma_lint.check(asm)
    assert len(found) == 1 and "after 0 states" in found[0]


def test_enough_states_are_clean():
    asm = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	s_nop 7
	v_add_f32_e32 v12, v1, v13
"""
    assert mfma_lint.check(asm) == []


def test_accumulator_chaining_is_clean_and_ab_read_is_reported():
    chain = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	v_mfma_f32_16x16x32_f16 v[0:3], v[14:17], v[18:21], v[0:3]
	s_nop 7
	global_store_dwordx4 v[30:31], v[0:3], off
"""
    assert mfma_lint.check(chain) == []
    ab = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	v_mfma_f32_16x16x32_f16 v[20:23], v[0:3], v[8:11], v[20:23]
"""
    assert any("A/B operand" in f for f in mfma_lint.check(ab))


def test_store_of_result_counts_as_a_read():
    asm = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	v_mov_b32_e32 v40, 0
	global_store_dwordx4 v[30:31], v[0:3], off
"""
    found = mfma_lint.check(asm)
    assert len(found) == 1 and "after 1 states" in found[0]


def test_scan_stops_at_an_unconditional_branch():
    asm = HEAD + """
	v_mfma_f32_16x16x4_f32 a[0:3], v1, v2, a[0:3]
	s_branch .LBB0_2
.LBB0_1:
	v_accvgpr_read_b32 v51, a3
"""
    assert mfma_lint.check(asm) == []
    fall = HEAD + """
	v_mfma_f32_16x16x4_f32 a[0:3], v1, v2, a[0:3]
	s_cbranch_scc1 .LBB0_2
.LBB0_1:
	v_accvgpr_read_b32 v51, a3
"""
    assert len(mfma_lint.check(fall)) == 1


def test_threshold_follows_the_instruction():
    """7 states after a 16-bit 16x16x32 and 9 after the fp32 16x16x4 are too
    few (the compiler leaves at least 8 and 10 on every straight-line path)."""
    f16 = HEAD + """
	v_mfma_f32_16x16x32_f16 v[0:3], v[4:7], v[8:11], v[0:3]
	s_nop 6
	v_add_f32_e32 v12, v1, v13
"""
    assert any("after 7 states" in f for f in mfma_lint.check(f16))
    f32 = HEAD + """
	v_mfma_f32_16x16x4_f32 a[0:3], v1, v2, a[0:3]
	s_nop 7
	v_mov_b32_e32 v40, 0
	v_accvgpr_read_b32 v51, a3
"""
    assert any("after 9 states" in f for f in mfma_lint.check(f32))
    ok = f32.replace("s_nop 7", "s_nop 7\n\tv_mov_b32_e32 v41, 0")
    assert mfma_lint.check(ok) == []
