"""The build's check of the device assembly (paper_2609_37007_amd/build_ext.py,
inflight_reads): an inline-assembly device-coherent load is invisible to the
compiler's wait insertion, so no instruction may touch its destination
registers before the s_waitcnt vmcnt(0) of its vm_wait."""
import pytest

from paper_2609_37007_amd.build_ext import inflight_reads

HEAD = "_ZN5rvqsd6kernelEv:  ; @kernel\n"


def asm(*lines):
    return HEAD + "\n".join("\t" + l for l in lines) + "\n"


def test_copy_before_wait_is_found():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "v_mov_b32_e32 v40, v32",
            "s_waitcnt vmcnt(0)")
    bad = inflight_reads(a)
    assert len(bad) == 1 and "v_mov_b32_e32 v40, v32" in bad[0][1]


def test_overwrite_before_wait_is_found():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "v_mov_b32_e32 v34, 0",
            "s_waitcnt vmcnt(0)")
    assert len(inflight_reads(a)) == 1


def test_register_range_operand_is_found():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "v_mfma_f32_16x16x32_bf16 v[0:3], v[30:33], v[4:7], v[0:3]",
            "s_waitcnt vmcnt(0)")
    assert len(inflight_reads(a)) == 1


def test_use_after_wait_is_clean():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "global_load_dwordx4 v[36:39], v[4:5], off sc1",
            "v_add_u32_e32 v1, v2, v3",
            "s_waitcnt vmcnt(0)",
            "v_mov_b32_e32 v40, v32",
            "v_and_b32_e32 v41, 1, v39")
    assert inflight_reads(a) == []


def test_partial_wait_does_not_clear():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "s_waitcnt vmcnt(1)",
            "v_mov_b32_e32 v40, v33",
            "s_waitcnt vmcnt(0)")
    assert len(inflight_reads(a)) == 1


def test_compiler_tracked_loads_and_other_functions_are_ignored():
    a = asm("buffer_load_dwordx4 v[32:35], v1, s[0:3], 0 offen sc1",
            "global_load_dwordx2 v[36:37], v[2:3], off sc1",
            "v_mov_b32_e32 v40, v32",
            "v_mov_b32_e32 v41, v36")
    assert inflight_reads(a) == []
    two = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1", "s_endpgm") + \
        "_ZN5rvqsd7kernel2Ev:\n\tv_mov_b32_e32 v40, v32\n"
    assert inflight_reads(two) == []


def test_comments_and_labels_are_not_instructions():
    a = asm("global_load_dwordx4 v[32:35], v[2:3], off sc1",
            "; v_mov_b32_e32 v40, v32",
            ".LBB0_3:",
            "s_waitcnt vmcnt(0)")
    assert inflight_reads(a) == []
