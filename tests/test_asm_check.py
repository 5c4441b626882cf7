"""The build-time check of inline-assembly LDS reads (asm_check.py): on
synthetic assembly it accepts reads whose registers stay untouched until a
wait that completes them (also across a loop back edge or after later LDS
reads with lgkmcnt(N)) and rejects copies, spills, uses on a path that skips
the wait and waits that leave the read in flight; the build's report lists
every kernel that waits for such reads in a later statement."""
import json
import os

import pytest

from paper_1802_00930_amd import asm_check, build

KERNEL = "_Zk:\n%s\n\ts_endpgm\n.Lfunc_end0:\n"


def problems(body):
    rep = asm_check.check_text(KERNEL % body)
    return rep["_Zk"]


def test_read_wait_use_is_clean():
    assert problems("\tds_read_b128 v[4:7], v1\n\tv_add_u32 v9, v2, v3\n\ts_waitcnt lgkmcnt(0)\n"
                    "\tv_mfma_i32_32x32x32_i8 v[16:31], v[4:7], v[8:11], 0") == []


def test_copy_before_wait_is_flagged():
    p = problems("\tds_read_b128 v[4:7], v1\n\tv_mov_b32 v20, v5\n\ts_waitcnt lgkmcnt(0)")
    assert len(p) == 1 and "v_mov_b32 v20, v5" in p[0]


def test_spill_before_wait_is_flagged():
    assert problems("\tds_read2_b64 v[4:7], v1 offset1:1\n\tscratch_store_dword off, v6, s0\n"
                    "\ts_waitcnt lgkmcnt(0)")


def test_overwrite_before_wait_is_flagged():
    assert problems("\tds_read_b64 v[4:5], v1\n\tv_mov_b32 v4, 0\n\ts_waitcnt lgkmcnt(0)")


def test_wait_after_loop_back_edge_is_clean():
    body = ("\ts_mov_b32 s4, 8\n\tds_read_b128 v[4:7], v1\n.LBB0_1:\n\ts_waitcnt lgkmcnt(0)\n"
            "\tv_mfma_i32_32x32x32_i8 v[16:31], v[4:7], v[8:11], v[16:31]\n"
            "\tds_read_b128 v[4:7], v2\n\tv_add_u32 v9, v9, 1\n\ts_add_i32 s4, s4, -1\n"
            "\ts_cmp_lg_u32 s4, 0\n\ts_cbranch_scc1 .LBB0_1\n\ts_waitcnt lgkmcnt(0)")
    assert problems(body) == []


def test_branch_around_the_wait_is_flagged():
    body = ("\tds_read_b128 v[4:7], v1\n\ts_cbranch_scc1 .LBB0_2\n\ts_waitcnt lgkmcnt(0)\n"
            ".LBB0_2:\n\tv_add_u32 v9, v4, 1")
    assert problems(body)


def test_lgkmcnt_counts_later_lds_reads():
    clean = ("\tds_read_b128 v[4:7], v1\n\tds_read_b128 v[12:15], v2\n\ts_waitcnt lgkmcnt(1)\n"
             "\tv_add_u32 v9, v4, 1\n\ts_waitcnt lgkmcnt(0)\n\tv_add_u32 v9, v12, 1")
    assert problems(clean) == []
    early = ("\tds_read_b128 v[4:7], v1\n\tds_read_b128 v[12:15], v2\n\ts_waitcnt lgkmcnt(1)\n"
             "\tv_add_u32 v9, v12, 1")
    assert problems(early)
    vm_only = "\tds_read_b128 v[4:7], v1\n\ts_waitcnt vmcnt(0)\n\tv_add_u32 v9, v4, 1"
    assert problems(vm_only)


def test_build_report_covers_every_split_read_kernel():
    if not os.path.exists(build.ASM_REPORT):
        pytest.skip("library not built")
    rep = json.load(open(build.ASM_REPORT))
    for src, table in build.SPLIT_READ_KERNELS.items():
        assert src in rep
        for frag in table:
            assert any(frag in k for k in rep[src]["kernels_checked"]), (src, frag)
        assert rep[src]["out_of_use"] == [], rep[src]


def test_later_lds_read_may_reuse_registers_but_not_read_them():
    ok = ("\tds_read2_b64 v[4:7], v1 offset1:1\n\tds_read_b64 v[4:5], v2\n\ts_waitcnt lgkmcnt(0)\n"
          "\tv_add_u32 v9, v4, v6")
    assert problems(ok) == []
    partly = "\tds_read2_b64 v[4:7], v1 offset1:1\n\tds_read_b64 v[4:5], v2\n\tv_add_u32 v9, v6, 1"
    assert problems(partly)
    addr = "\tds_read_b64 v[4:5], v1\n\tds_read_b64 v[8:9], v4\n\ts_waitcnt lgkmcnt(0)"
    assert problems(addr)
