"""The build's scan of the device assembly for DPP hazards (host logic)."""
from paper_2609_39361_amd.build import scan_dpp_hazards as scan

DPP = "v_fmac_f32_dpp v1, v3, v2 row_newbcast:0 row_mask:0xf bank_mask:0xf"


def test_vgpr_write_right_before_dpp():
    assert scan("v_mov_b32 v3, v4\n" + DPP + "\n")


def test_wide_write_overlapping_src():
    assert scan("v_mov_b64 v[2:3], v[8:9]\ns_nop 0\n" + DPP + "\n")


def test_two_wait_states_are_enough():
    assert not scan("v_mov_b32 v3, v4\ns_nop 1\n" + DPP + "\n")
    assert not scan("v_mov_b32 v3, v4\nv_add_f32 v7, v8, v9\nv_add_f32 v7, v8, v9\n" + DPP + "\n")


def test_write_of_other_vgpr_is_fine():
    assert not scan("v_mov_b32 v2, v4\n" + DPP + "\n")


def test_load_write_is_not_a_valu_hazard():
    assert not scan("global_load_dwordx4 v[0:3], v[10:11], off\ns_waitcnt vmcnt(0)\n" + DPP + "\n")


def test_exec_write_needs_five():
    assert scan("v_cmpx_gt_f32 exec, v5, v6\ns_nop 3\n" + DPP + "\n")
    assert not scan("v_cmpx_gt_f32 exec, v5, v6\ns_nop 4\n" + DPP + "\n")


def test_hazard_across_loop_back_edge():
    asm = ".LBB0_1:\n" + DPP + "\ns_nop 3\nv_mov_b32 v3, v9\ns_cbranch_scc1 .LBB0_1\ns_endpgm\n"
    assert scan(asm)


def test_hazard_through_forward_branch():
    asm = "v_mov_b32 v3, v9\ns_cbranch_vccz .LBB0_2\ns_nop 7\n.LBB0_2:\n" + DPP + "\n"
    assert scan(asm)
    asm_ok = "v_mov_b32 v3, v9\ns_nop 1\ns_cbranch_vccz .LBB0_2\ns_nop 7\n.LBB0_2:\n" + DPP + "\n"
    assert not scan(asm_ok)


def test_unconditional_branch_cuts_fall_through():
    asm = "v_mov_b32 v3, v9\ns_branch .LBB0_3\n.LBB0_2:\n" + DPP + "\ns_endpgm\n.LBB0_3:\ns_nop 4\ns_branch .LBB0_2\n"
    assert not scan(asm)
