"""The library's log2 table (generated with integer arithmetic by
paper_2608_18147_amd/csrc/gen_log2_table.py) and the oracle's (mpmath) are
built independently; both claim correctly rounded entries, so they must agree
bit for bit."""
import os
import re

from oracle.log2_table import OFF_HI, TABLE_BITS, build_table

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_table_matches_oracle_table():
    src = open(os.path.join(ROOT, "paper_2608_18147_amd", "csrc", "log2_table.inc")).read()
    assert int(re.search(r"ECASQ_LOG2_OFF_HI 0x([0-9A-F]+)u", src).group(1), 16) == OFF_HI
    assert int(re.search(r"ECASQ_LOG2_BITS (\d+)", src).group(1)) == TABLE_BITS
    rows = re.findall(r"\{(-?0x[0-9a-fp.+-]+), (-?0x[0-9a-fp.+-]+)\}", src)
    lib = [(float.fromhex(a), float.fromhex(b)) for a, b in rows]
    invc, lc = build_table()
    assert len(lib) == len(invc) == 1 << TABLE_BITS
    for (a, b), c, d in zip(lib, invc, lc):
        assert a == c and b == d
