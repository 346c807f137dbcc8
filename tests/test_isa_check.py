"""The build-time check of untracked inline-asm LDS reads (isa_check) on small assembly
listings with known answers, and on the attention assembly of the last build if present."""
import os

import pytest

from paper_2608_29748_amd import isa_check

HEAD = "_ZN2rt4kernEv:                  ; @k\n"
TAIL = "\ts_endpgm\n.Lfunc_end0:\n"


def listing(body: str) -> str:
    return HEAD + body + TAIL


def asm_read(dst: str, addr: str = "v0") -> str:
    return f"\t;;#ASMSTART\n\tds_read_b128 {dst}, {addr}\n\t;;#ASMEND\n"


def test_wait_then_use_is_clean():
    src = listing(asm_read("v[4:7]") + "\ts_waitcnt lgkmcnt(0)\n\tv_add_f32_e32 v8, v4, v5\n")
    assert isa_check.checked_kernels(src) == ["_ZN2rt4kernEv"]
    assert isa_check.check(src) == []


def test_use_before_wait_is_flagged():
    src = listing(asm_read("v[4:7]") + "\tv_add_f32_e32 v8, v4, v5\n\ts_waitcnt lgkmcnt(0)\n")
    assert len(isa_check.check(src)) == 1


def test_overwrite_before_wait_is_flagged():
    # a register reused for another value while the read may still land in it
    src = listing(asm_read("v[4:7]") + "\tv_mov_b32_e32 v6, 0\n\ts_waitcnt lgkmcnt(0)\n")
    assert isa_check.check(src) == ["_ZN2rt4kernEv: v_mov_b32_e32 v6, 0"]


def test_partial_wait_counts_later_lds_operations():
    # lgkmcnt(1) leaves only the last LDS operation outstanding: the earlier read is done
    ok = listing(asm_read("v[4:7]") + asm_read("v[8:11]") + "\ts_waitcnt lgkmcnt(1)\n\tv_mov_b32_e32 v4, 0\n"
                 "\ts_waitcnt lgkmcnt(0)\n")
    assert isa_check.check(ok) == []
    bad = listing(asm_read("v[4:7]") + asm_read("v[8:11]") + "\ts_waitcnt lgkmcnt(1)\n\tv_mov_b32_e32 v8, 0\n"
                  "\ts_waitcnt lgkmcnt(0)\n")
    assert len(isa_check.check(bad)) == 1


def test_path_that_skips_the_wait_is_flagged():
    # the wait sits on one arm of a branch only; the join reads the register
    body = (asm_read("v[4:7]") + "\ts_cbranch_scc1 .LBB0_2\n"
            "\ts_waitcnt lgkmcnt(0)\n"
            ".LBB0_2:\n\tv_add_f32_e32 v8, v4, v5\n\ts_waitcnt lgkmcnt(0)\n")
    assert len(isa_check.check(listing(body))) == 1
    body_ok = (asm_read("v[4:7]") + "\ts_waitcnt lgkmcnt(0)\n\ts_cbranch_scc1 .LBB0_2\n"
               "\tv_mov_b32_e32 v9, 0\n"
               ".LBB0_2:\n\tv_add_f32_e32 v8, v4, v5\n")
    assert isa_check.check(listing(body_ok)) == []


def test_loop_back_edge_carries_pending_reads():
    # the read at the loop's end is used at its head before any wait
    body = (".LBB0_1:\n\tv_add_f32_e32 v8, v4, v5\n" + asm_read("v[4:7]") +
            "\ts_cbranch_scc1 .LBB0_1\n\ts_waitcnt lgkmcnt(0)\n")
    assert len(isa_check.check(listing(body))) == 1


def test_kernels_without_asm_reads_are_not_checked():
    src = listing("\tds_read_b128 v[4:7], v0\n\tv_add_f32_e32 v8, v4, v5\n")
    assert isa_check.checked_kernels(src) == []
    assert isa_check.check(src) == []


def test_last_built_attention_assembly():
    path = os.path.join(os.path.dirname(isa_check.__file__), "_build", "attn.s")
    if not os.path.exists(path):
        pytest.skip("no build of the attention assembly in this tree")
    with open(path) as fh:
        asm = fh.read()
    assert isa_check.checked_kernels(asm)
    assert isa_check.check(asm) == []
