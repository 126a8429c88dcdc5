"""The build-time scan for the SCC miscompile (paper_2608_04991_amd/isa_check.py)."""
from paper_2608_04991_amd import isa_check

BAD = """_ZN3fooEv:
\ts_add_u32 s24, s30, s14
\ts_addc_u32 s23, s23, s15
\ts_and_b32 s25, s23, 0xffff
\ts_cselect_b32 s26, 0, s44
\ts_endpgm
"""

GOOD = """_ZN3fooEv:
\ts_add_u32 s24, s30, s14
\ts_addc_u32 s23, s23, s15
\ts_and_b32 s25, s23, 0xffff
\ts_and_b64 s[28:29], vcc, exec
\ts_cselect_b32 s26, 0, s44
\ts_cmp_lt_u32 s2, s3
\ts_cbranch_scc1 .LBB0_2
.LBB0_1:
\ts_cselect_b32 s4, 1, 0
\ts_endpgm
"""


def test_flags_a_select_after_an_address_mask():
    bad = isa_check.scan(BAD)
    assert len(bad) == 1 and "s_cselect_b32 s26, 0, s44" in bad[0]


def test_accepts_predicates_and_block_boundaries():
    assert isa_check.scan(GOOD) == []
