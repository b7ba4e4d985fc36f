"""The build's check for vector stores whose data registers the next
instruction overwrites (a store of more than 64 bits reads its data over two
cycles): it flags the sequence that corrupted outputs on gfx950 and accepts
the safe forms."""

from paper_2606_05613_amd.build import store_data_overwrites


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
