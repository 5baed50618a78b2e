"""The build's assembly check for untracked loads (paper_2606_19667_amd/asm_check.py)
on hand-written gfx9 snippets."""
import pytest

from paper_2606_19667_amd import asm_check


def _fn(body: str) -> str:
    return "k:\n" + body + "\n\ts_endpgm\n.Lfunc_end0:\n"


LOAD = "\t;;#ASMSTART\n\tglobal_load_dword v10, v[0:1], off\n\t;;#ASMEND\n"


def _hazards(body):
    return asm_check.hazards(_fn(body).split("\n"))


def test_read_before_any_wait_is_reported():
    assert _hazards(LOAD + "\tv_mov_b32_e32 v2, v10\n")


def test_write_before_the_wait_is_reported():
    assert _hazards(LOAD + "\tv_mov_b32_e32 v10, 0\n\ts_waitcnt vmcnt(0)\n")


def test_wait_that_covers_the_load_clears_it():
    body = LOAD + "".join(f"\tglobal_load_lds_dwordx4 v{20 + i}, s[4:5]\n" for i in range(4))
    assert not _hazards(body + "\ts_waitcnt vmcnt(4)\n\tv_readfirstlane_b32 s6, v10\n")
    # vmcnt(4) with only 3 younger memory instructions does not cover it
    body3 = LOAD + "".join(f"\tglobal_load_lds_dwordx4 v{20 + i}, s[4:5]\n" for i in range(3))
    assert _hazards(body3 + "\ts_waitcnt vmcnt(4)\n\tv_readfirstlane_b32 s6, v10\n")


def test_every_path_is_followed():
    body = LOAD + ("\ts_cbranch_scc1 .LBB0_2\n\ts_waitcnt vmcnt(0)\n.LBB0_2:\n"
                   "\tv_readfirstlane_b32 s6, v10\n")
    assert _hazards(body)
    body_ok = LOAD + ("\ts_waitcnt vmcnt(0)\n\ts_cbranch_scc1 .LBB0_2\n\ts_nop 0\n.LBB0_2:\n"
                      "\tv_readfirstlane_b32 s6, v10\n")
    assert not _hazards(body_ok)


def test_barrier_ends_the_window_and_waited_asm_loads_are_tracked():
    assert not _hazards(LOAD + "\ts_barrier\n\tv_readfirstlane_b32 s6, v10\n")
    waited = ("\t;;#ASMSTART\n\tglobal_load_dwordx4 v[10:13], v[0:1], off\n\ts_waitcnt vmcnt(0)\n"
              "\t;;#ASMEND\n\tv_mov_b32_e32 v2, v10\n")
    assert not _hazards(waited)


def test_check_raises_with_the_function_name():
    text = _fn(LOAD + "\tv_mov_b32_e32 v2, v10\n").replace("k:", "my_suffix_prefill_attn_kernel:")
    with pytest.raises(RuntimeError, match="my_suffix_prefill_attn_kernel"):
        asm_check.check(text)
    with pytest.raises(RuntimeError, match="no function"):
        asm_check.check(_fn("\ts_nop 0\n"))


def test_flag_tests_on_a_lane_mask_follow_both_directions():
    # if (F) { load } ; if (!F) { use } with F a per-lane compare: some lanes may
    # take each arm, so the use after the load is reported
    body = ("\tv_cmp_gt_i32_e64 s[12:13], 3, v1\n\ts_and_b64 vcc, exec, s[12:13]\n\ts_cbranch_vccz .LBB0_2\n"
            + LOAD + ".LBB0_2:\n\ts_andn2_b64 vcc, exec, s[12:13]\n\ts_cbranch_vccz .LBB0_3\n"
            "\tv_readfirstlane_b32 s6, v10\n.LBB0_3:\n\ts_waitcnt vmcnt(0)\n")
    assert _hazards(body)


def test_flag_set_to_a_constant_is_known():
    # F = -1; if (c) { F = 0; load }; if (F) { use }: the use never follows the load
    body = ("\ts_mov_b64 s[12:13], -1\n\ts_cbranch_scc1 .LBB0_2\n\ts_mov_b64 s[12:13], 0\n" + LOAD +
            ".LBB0_2:\n\ts_and_b64 vcc, exec, s[12:13]\n\ts_cbranch_vccz .LBB0_3\n"
            "\tv_readfirstlane_b32 s6, v10\n.LBB0_3:\n\ts_waitcnt vmcnt(0)\n")
    assert not _hazards(body)
    assert _hazards(body.replace("s_mov_b64 s[12:13], 0\n", "s_mov_b64 s[12:13], s[4:5]\n"))
    # the flag written in between by something else: both directions again
    body_w = body.replace(".LBB0_2:\n", ".LBB0_2:\n\ts_cselect_b64 s[12:13], -1, 0\n")
    assert _hazards(body_w)
    # the other constant: the use follows the load
    assert _hazards(body.replace("s_mov_b64 s[12:13], 0\n", "s_mov_b64 s[12:13], -1\n", 1).replace(
        "\ts_mov_b64 s[12:13], -1\n\ts_cbranch_scc1", "\ts_mov_b64 s[12:13], 0\n\ts_cbranch_scc1"))


SLOAD = "\t;;#ASMSTART\n\ts_load_dwordx2 s[12:13], s[4:5], 0x0\n\t;;#ASMEND\n"


def test_scalar_load_destination_use_before_lgkmcnt0_is_reported():
    # a read (copy) and a write of the destination before the wait
    assert _hazards(SLOAD + "\ts_mov_b32 s20, s13\n\ts_waitcnt lgkmcnt(0)\n")
    assert _hazards(SLOAD + "\ts_add_u32 s12, s12, 4\n")
    # a vector wait, or a partial lgkm wait, does not cover a scalar load
    assert _hazards(SLOAD + "\ts_waitcnt vmcnt(0)\n\tv_mov_b32_e32 v2, s12\n")
    assert _hazards(SLOAD + "\ts_waitcnt lgkmcnt(1)\n\tv_mov_b32_e32 v2, s12\n")
    # nor does a barrier without the wait
    assert _hazards(SLOAD + "\ts_barrier\n\tv_mov_b32_e32 v2, s12\n")


def test_scalar_load_covered_by_lgkmcnt0_is_clear():
    assert not _hazards(SLOAD + "\ts_mov_b32 s20, s14\n\ts_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier\n"
                                "\tv_mov_b32_e32 v2, s12\n\ts_add_u32 s12, s12, 4\n")
    # other registers may be used meanwhile, and the paths all pass the wait
    body = SLOAD + ("\ts_cbranch_scc1 .LBB0_2\n\ts_mov_b32 s30, 1\n.LBB0_2:\n"
                    "\ts_waitcnt lgkmcnt(0)\n\ts_mov_b32 s20, s13\n")
    assert not _hazards(body)
