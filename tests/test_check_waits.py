"""The build's check of the BF6 GEMM's hand-ordered vector loads
(check_waits.py), on hand-written assembly: along every control-flow path it
must flag each touch of a load's destination registers that no vmcnt wait has
retired, and nothing else."""

import pytest

from paper_2609_33601_amd import check_waits

HEAD = "_ZN2jq12_GLOBAL__N_119w4a4_f6_gemm_kernelILi8EEEvPKh:\n"
TAIL = "\ts_endpgm\n"


def run(body):
    return check_waits.hazards(check_waits.kernels(HEAD + body + TAIL, "w4a4_f6_gemm_kernel")[0][1])


def test_read_before_wait_is_flagged():
    found = run("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
                "\tv_mov_b32_e32 v8, v5\n")
    assert len(found) == 1 and "v_mov_b32_e32 v8, v5" in found[0][1]


def test_read_after_retiring_wait_is_clean():
    assert run("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
               "\ts_waitcnt vmcnt(0)\n"
               "\tv_mov_b32_e32 v8, v5\n") == []


def test_in_order_completion():
    # vmcnt(1) retires the older of two loads only
    body = ("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
            "\tbuffer_load_dwordx4 v[12:15], v0, s[0:3], s4 offen\n"
            "\ts_waitcnt vmcnt(1)\n")
    assert run(body + "\tv_mov_b32_e32 v8, v7\n") == []
    assert len(run(body + "\tv_mov_b32_e32 v8, v12\n")) == 1


def test_spill_of_pending_load_and_overwrite_are_flagged():
    # a scratch store of the registers (a spill) and a write into them both count
    assert len(run("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
                   "\tscratch_store_dwordx4 off, v[4:7], off\n")) == 1
    assert len(run("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
                   "\tv_mov_b32_e32 v6, 0\n")) == 1


def test_lds_dma_has_no_destination_registers():
    assert run("\ts_mov_b32 m0, s5\n"
               "\tbuffer_load_dwordx4 v4, s[0:3], s6 offen lds\n"
               "\tv_mov_b32_e32 v4, 1\n") == []


def test_loop_wrap():
    # a load at the bottom of the loop body, read at its top with no wait between
    body = (".LBB0_1:\n"
            "\tv_mov_b32_e32 v8, v4\n"
            "\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
            "\ts_cbranch_scc1 .LBB0_1\n")
    assert len(run(body)) >= 1
    # the same with the wait at the top of the loop is clean
    assert run(body.replace(".LBB0_1:\n", ".LBB0_1:\n\ts_waitcnt vmcnt(0)\n")) == []


def test_out_of_line_block_is_checked_where_it_runs():
    # a block placed after the load in the text but reached only from before it
    body = ("\ts_cbranch_scc1 .LBB0_9\n"
            ".LBB0_2:\n"
            "\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
            "\ts_waitcnt vmcnt(0)\n"
            "\ts_endpgm\n"
            ".LBB0_9:\n"
            "\tv_mov_b32_e32 v4, 1\n"
            "\ts_branch .LBB0_2\n")
    assert run(body) == []
    # reached from after the load instead: flagged
    body2 = ("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
             "\ts_cbranch_scc1 .LBB0_9\n"
             "\ts_waitcnt vmcnt(0)\n"
             "\ts_endpgm\n"
             ".LBB0_9:\n"
             "\tv_mov_b32_e32 v4, 1\n"
             "\ts_endpgm\n")
    assert len(run(body2)) == 1


def test_paths_merge_conservatively():
    # waited for on one path only: still pending where the paths meet
    body = ("\tbuffer_load_dwordx4 v[4:7], v0, s[0:3], s4 offen\n"
            "\ts_cbranch_scc1 .LBB0_3\n"
            "\ts_waitcnt vmcnt(0)\n"
            ".LBB0_3:\n"
            "\tv_mov_b32_e32 v8, v5\n")
    assert len(run(body)) == 1


def test_check_asm_raises_and_counts():
    with pytest.raises(RuntimeError, match="ordering check failed"):
        check_waits.check_asm(HEAD + "\tbuffer_load_dword v4, v0, s[0:3], 0 offen\n\tv_add_u32_e32 v1, v4, v2\n" + TAIL)
    assert check_waits.check_asm(HEAD + "\ts_nop 0\n" + TAIL) == 1
    with pytest.raises(RuntimeError, match="no kernel"):
        check_waits.check_asm("foo:\n\ts_endpgm\n")
