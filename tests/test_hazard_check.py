"""The build-time MFMA hazard checker flags the spacing violations it exists for, on small
hand-written gfx950 assembly, and accepts correctly spaced code."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2608_25683_amd import hazard_check as H  # noqa: E402

MF = "v_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], a[0:3], v[0:15]"


def kinds(lines):
    return [b[0] for b in H.check(lines)]


def test_valu_read_right_after_mfma_is_flagged():
    assert kinds([MF, "v_add_f32_e32 v20, v3, v21"]) == ["R1 mfma->other"]


def test_twelve_wait_states_are_enough():
    assert kinds([MF, "s_nop 11", "v_add_f32_e32 v20, v3, v21"]) == []
    assert kinds([MF, "s_nop 10", "v_add_f32_e32 v20, v3, v21"]) == ["R1 mfma->other"]


def test_overwrite_of_pending_result_is_flagged():
    # a load into a register the MFMA has not written yet (write after write)
    assert kinds([MF, "ds_read_b64 v[4:5], v30"]) == ["R1 mfma->other"]


def test_accumulate_chain_is_allowed():
    assert kinds([MF, MF, "s_nop 11", "v_mov_b32_e32 v40, v0"]) == []


def test_operand_written_by_valu_needs_two_wait_states():
    mf = "v_mfma_f32_32x32x16_bf16 a[0:15], v[16:19], v[20:23], a[0:15]"
    assert kinds(["v_cvt_pk_bf16_f32 v21, v1, v2", mf]) == ["R2 valu->mfma"]
    assert kinds(["v_cvt_pk_bf16_f32 v21, v1, v2", "s_nop 1", mf]) == []


def test_branches_are_followed():
    lines = [MF, "s_cbranch_scc1 .LBB0_2", "s_nop 15", ".LBB0_2:", "v_mov_b32_e32 v40, v5"]
    assert kinds(lines) == ["R1 mfma->other"]


def test_valu_write_into_pending_result_across_a_block_is_flagged():
    # an MFMA whose result has no reader, then the next block reuses one of its registers
    lines = [MF, "s_branch .LBB0_3", ".LBB0_3:", "v_or_b32_e32 v4, s6, v0"]
    assert kinds(lines) == ["R1 mfma->other"]
    assert kinds([MF, "s_nop 11", "s_branch .LBB0_3", ".LBB0_3:", "v_or_b32_e32 v4, s6, v0"]) == []
