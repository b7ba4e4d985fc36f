"""The build's checks of the generated gfx950 code: vector stores whose data
registers the next instruction overwrites (a store of more than 64 bits
reads its data over two cycles), flagged in the sequence that corrupted
outputs on gfx950 and accepted in the safe forms; and the order of the
pipelined kernel's cross-workgroup hand-offs (publish point, then the flag
or counter; poll loop, then the observe point, then the data loads)."""

import os

import pytest

from paper_2606_05613_amd.build import BUILD, handoff_order_violations, store_data_overwrites


def _check(tmp_path, text):
    p = tmp_path / "k.s"
    p.write_text(text)
    return store_data_overwrites(str(p))


def test_flags_wide_store_followed_by_data_overwrite(tmp_path):
    asm = """\tbuffer_store_dwordx4 v[146:149], v169, s[56:59], s26 offen nt
\tv_cndmask_b32_e64 v146, 0, 1, s[14:15]
\tglobal_store_dwordx4 v[2:3], v[8:11], off
\tv_mov_b32_e32 v10, v1
"""
    hits = _check(tmp_path, asm)
    assert len(hits) == 2 and hits[0][0] == 1 and hits[1][0] == 3


def test_accepts_narrow_stores_and_unrelated_writes(tmp_path):
    asm = """\tbuffer_store_dwordx2 v[146:147], v169, s[56:59], s26 offen nt
\tv_mov_b32_e32 v146, v18
\tbuffer_store_dwordx4 v[146:149], v169, s[56:59], s26 offen nt
\tv_mov_b32_e32 v150, v18
\tglobal_store_dwordx4 v[2:3], v[8:11], off ; comment v8
\ts_nop 0
\tv_mov_b32_e32 v8, v1
"""
    assert _check(tmp_path, asm) == []


# ---- cross-workgroup hand-off order (publish / observe points) ----

GOOD = """_ZN5bkmoo13hybrid_kernelILi4EEEv:
\tglobal_store_dwordx2 v1, v[2:3], s[4:5] sc1
\t;;#ASMSTART
\ts_waitcnt vmcnt(0) ; bkmoo publish
\t;;#ASMEND
\ts_add_u32 s14, s20, s14
\tglobal_atomic_add v17, v95, s[14:15]
.LBB0_20:
\tglobal_load_dword v2, v1, s[4:5] sc1
\ts_waitcnt vmcnt(0)
\ts_sleep 1
\ts_branch .LBB0_20
.LBB0_27:
\tglobal_atomic_or v17, v92, s[22:23]
\tds_write_b32 v93, v2
\t;;#ASMSTART
\t; bkmoo observe
\t;;#ASMEND
\tglobal_load_dword v3, v1, s[6:7] sc1
.Lfunc_end0:
"""


def _order(tmp_path, text):
    p = tmp_path / "h.s"
    p.write_text(text)
    return handoff_order_violations(str(p))


def test_handoff_order_accepts_publish_then_flag_and_observe_after_poll(tmp_path):
    assert _order(tmp_path, GOOD) == []
    flag = GOOD.replace("global_atomic_add v17, v95, s[14:15]", "global_store_dword v17, v95, s[14:15] sc1")
    assert _order(tmp_path, flag) == []


def test_handoff_order_flags_a_data_store_after_the_publish_point(tmp_path):
    bad = GOOD.replace("\ts_add_u32 s14, s20, s14\n", "\tglobal_store_dwordx2 v1, v[2:3], s[8:9] sc1\n")
    assert len(_order(tmp_path, bad)) == 1


def test_handoff_order_flags_a_block_between_publish_and_flag(tmp_path):
    bad = GOOD.replace("\ts_add_u32 s14, s20, s14\n", ".LBB0_16:\n")
    assert len(_order(tmp_path, bad)) == 1


def test_handoff_order_flags_a_load_hoisted_before_the_observe_point(tmp_path):
    bad = GOOD.replace("\tds_write_b32 v93, v2\n", "\tglobal_load_dword v3, v1, s[6:7] sc1\n")
    assert len(_order(tmp_path, bad)) == 1


def test_handoff_order_flags_missing_points(tmp_path):
    bad = GOOD.replace("bkmoo observe", "something else")
    assert len(_order(tmp_path, bad)) == 1
    no_loop = GOOD.replace("\ts_sleep 1\n", "")
    assert len(_order(tmp_path, no_loop)) == 1


@pytest.mark.parametrize("unit", ["hybrid", "refill"])
def test_built_cooperative_kernels_hand_off_in_order(unit):
    asm = os.path.join(BUILD, f"{unit}-hip-amdgcn-amd-amdhsa-gfx950.s")
    if not os.path.exists(asm):
        pytest.skip("library not built")
    assert handoff_order_violations(asm, f"{unit}_kernel") == []
