"""The build's check of the staged global->LDS loads' SGPR bases (no GPU).

build.staging_hazards scans gfx950 assembly for a VALU write of a base SGPR
fewer than 5 wait states before the global_load_lds that reads it, which the
compiler's hazard tracking does not see inside inline asm.
"""
import importlib.util
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_spec = importlib.util.spec_from_file_location("rl_build", os.path.join(ROOT, "paper_2607_20908_amd", "build.py"))
build = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(build)


def scan(text):
    return build.staging_hazards(text)


def test_valu_write_just_before_is_flagged():
    n, errs = scan("\tv_readfirstlane_b32 s28, v6\n\ts_mov_b32 s29, 0\n\ts_nop 0\n"
                   "\tglobal_load_lds_dwordx4 v13, s[28:29]\n")
    assert n == 1 and len(errs) == 1 and "2 wait states" in errs[0]


def test_five_wait_states_are_enough():
    n, errs = scan("\tv_readfirstlane_b32 s30, v6\n\ts_nop 4\n\tglobal_load_lds_dwordx4 v13, s[30:31]\n")
    assert n == 1 and errs == []


def test_salu_writer_after_the_valu_write_is_safe():
    # the last writer of the base decides: here an SALU op rewrites it
    n, errs = scan("\tv_readfirstlane_b32 s6, v8\n\ts_or_b64 s[6:7], s[6:7], s[4:5]\n\ts_nop 0\n"
                   "\tglobal_load_lds_dwordx4 v12, s[6:7]\n")
    assert errs == []


def test_carry_out_of_a_valu_op_is_a_write():
    n, errs = scan("\tv_mad_u64_u32 v[2:3], s[8:9], s4, v1, v[2:3]\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert len(errs) == 1


def test_writer_in_a_predecessor_block_is_flagged():
    # fall-through predecessor
    n, errs = scan("\tv_readfirstlane_b32 s8, v1\n.LBB0_3:\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert len(errs) == 1 and "LBB0_3" in errs[0]
    # branch predecessor only (the line before the label ends its block)
    n, errs = scan("\tv_readfirstlane_b32 s9, v1\n\ts_cbranch_scc1 .LBB0_3\n\ts_endpgm\n"
                   ".LBB0_3:\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert len(errs) == 1 and "1 wait states" in errs[0]   # the branch itself
    # the same with enough wait states on every path
    n, errs = scan("\tv_readfirstlane_b32 s9, v1\n\ts_nop 3\n\ts_cbranch_scc1 .LBB0_3\n\ts_endpgm\n"
                   ".LBB0_3:\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert errs == []


def test_one_bad_path_of_several_is_flagged():
    text = ("\ts_mov_b32 s8, 0\n\ts_cbranch_scc0 .LBB0_4\n\tv_readfirstlane_b32 s8, v1\n"
            ".LBB0_4:\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    n, errs = scan(text)
    assert len(errs) == 1 and "v_readfirstlane_b32 s8" in errs[0]


def test_kernel_entry_and_loops():
    # a path that starts at the kernel entry has no writer
    n, errs = scan("kern:\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert errs == []
    # a loop whose back edge carries a VALU write of the base
    n, errs = scan("\ts_mov_b64 s[8:9], 0\n.LBB0_1:\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n"
                   "\tv_readfirstlane_b32 s8, v1\n\ts_cbranch_scc1 .LBB0_1\n\ts_endpgm\n")
    assert len(errs) == 1


def test_valu_write_of_m0_is_flagged():
    n, errs = scan("\tv_readfirstlane_b32 m0, v3\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert len(errs) == 1
    n, errs = scan("\ts_mov_b32 m0, s3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 v12, s[8:9]\n")
    assert errs == []


def test_vgpr_base_and_off_form():
    assert len(scan("\tglobal_load_lds_dwordx4 v12, v[8:9]\n")[1]) == 1
    n, errs = scan("\tv_add_u32_e32 v3, 1, v3\n\tglobal_load_lds_dwordx4 v[2:3], off\n")
    assert n == 1 and errs == []


@pytest.mark.parametrize("src", build.STAGING_ASM)
def test_built_kernels_are_clean(src):
    path = os.path.join(build.BUILD, os.path.splitext(src)[0] + ".gfx950.s")
    if not os.path.exists(path):
        pytest.skip("not built")
    with open(path) as f:
        n, errs = scan(f.read())
    assert n > 0 and errs == [], errs[:5]
