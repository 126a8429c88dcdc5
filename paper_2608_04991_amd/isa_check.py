"""Build-time check of the gfx950 assembly of librac for one known miscompile.

The ROCm 7.2 compiler's pre-emit peephole pass can delete an
``s_and_b64 vcc, vcc, exec`` whose SCC result a later ``s_cselect`` still
reads (seen when a uniform 64-bit comparison was made on the vector unit and
also feeds a ``s_cbranch_vccnz``).  The select then reads an SCC left by an
unrelated arithmetic instruction.  This scan flags every SCC consumer whose
nearest SCC writer in the same basic block is such an arithmetic instruction;
the kernels are written so that none exists.

  python -m paper_2608_04991_amd.isa_check FILE.s
"""
from __future__ import annotations

import re
import sys

_WRITER = re.compile(
    r"^\s+(s_add_u32|s_add_i32|s_sub_u32|s_sub_i32|s_addc_u32|s_subb_u32"
    r"|s_(and|or|xor|andn2|orn2|nand|nor|xnor|not)_b(32|64)|s_(lshl|lshr|ashr)_b(32|64)"
    r"|s_lshl[1-4]_add_u32|s_bfe_[iu](32|64)|s_(min|max)_[iu]32|s_cmp\w*|s_bitcmp\w*"
    r"|s_abs_i32|s_absdiff_i32|s_bcnt[01]_i32_b(32|64)|s_\w+_saveexec_b64|s_\w+_wrexec_b64)\s")
_CONSUMER = re.compile(r"^\s+(s_cselect_b(32|64)|s_cbranch_scc[01]|s_cmovk_i32|s_cmov_b(32|64))\s")
_ARITH = re.compile(
    r"^\s+(s_add_u32|s_add_i32|s_sub_u32|s_sub_i32|s_addc_u32|s_subb_u32|s_(lshl|lshr|ashr)_b(32|64)"
    r"|s_lshl[1-4]_add_u32|s_bfe_\w+|s_abs_i32|s_absdiff_i32|s_bcnt\w+"
    r"|s_and_b32\s+\S+,\s*\S+,\s*0xffff$)")


def scan(text: str) -> list[str]:
    bad, func, last = [], None, None
    for i, line in enumerate(text.split("\n"), 1):
        if re.match(r"^_Z\S+:", line):
            func, last = line.split(":")[0], None
        if re.match(r"^\.LBB|^; %bb", line):
            last = None
        if _CONSUMER.match(line) and last is not None and _ARITH.match(last[1]):
            bad.append(f"{func} line {i}: {last[1].strip()} -> {line.strip()}")
        if _WRITER.match(line):
            last = (i, line)
    return bad


if __name__ == "__main__":
    found = scan(open(sys.argv[1]).read())
    print("\n".join(found) if found else "no SCC read after an arithmetic SCC write")
    sys.exit(1 if found else 0)
