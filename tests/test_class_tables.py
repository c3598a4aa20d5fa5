"""The library's generated class tables against the oracle's classes (CPU only).

``csrc/gen_class_table.py`` probes the engine and writes the two-level tables
the kernels stage in LDS; the oracle reads its own probe files.  The two
derivations are compared here for every Unicode scalar value, so that a kernel
table can never drift from what the oracle (and its pins) see.  The
DeepSeek-style kernel also computes ASCII classes without the table; that
formula is written out again here and checked against the table.
"""

import os
import re

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_29678_amd", "csrc")


def _arrays(name, *arrays):
    with open(os.path.join(CSRC, name)) as f:
        src = f.read()
    out = []
    for a in arrays:
        m = re.search(a + r"\[\d+\][^=]*=\s*\{([^}]*)\}", src)
        out.append([int(x) for x in m.group(1).replace("\n", "").split(",") if x.strip()])
    return out


def _four_bit(l1, l2, cp):
    return (l2[l1[cp >> 8] * 128 + ((cp & 255) >> 1)] >> ((cp & 1) * 4)) & 15


def _oracle_deepseek_class(cp):
    from oracle.classes import L, N, W, char_class, is_mark, is_punct_or_symbol
    from oracle.pretok import in_kana_cjk

    c = char_class(cp)
    if in_kana_cjk(cp):
        return 10 if c == L else 11 if is_mark(cp) else 12 if is_punct_or_symbol(cp) else 13
    if cp in (10, 13):
        return 9
    if cp == 32:
        return 7
    if c == W:
        return 8
    if c == N:
        return 4
    if c == L:
        return 1 if cp < 128 else 2
    if is_mark(cp):
        return 3
    if is_punct_or_symbol(cp):
        return 5 if cp < 128 else 6
    return 0


def test_deepseek_table_equals_oracle_classes():
    l1, l2 = _arrays("class_table_deepseek.inc", "TT_DS_L1", "TT_DS_L2")
    bad = [cp for cp in range(0x110000) if not 0xD800 <= cp <= 0xDFFF
           and _four_bit(l1, l2, cp) != _oracle_deepseek_class(cp)]
    assert bad == [], bad[:10]


def test_deepseek_ascii_formula_equals_table():
    l1, l2 = _arrays("class_table_deepseek.inc", "TT_DS_L1", "TT_DS_L2")

    def formula(cp):  # ds_ascii_class in tt_deepseek.h
        if 0 <= (cp | 32) - ord("a") < 26:
            return 1
        if 0 <= cp - ord("0") < 10:
            return 4
        if cp in (10, 13):
            return 9
        if cp == 32:
            return 7
        if cp in (9, 11, 12):
            return 8
        if 33 <= cp < 127:
            return 5
        return 0

    assert [formula(cp) for cp in range(128)] == [_four_bit(l1, l2, cp) for cp in range(128)]


def test_o200k_table_equals_oracle_classes():
    from oracle.classes import BO, LO, MK, UP, L, N, W, o200k_class

    l1, l2 = _arrays("class_table_o200k.inc", "TT_O2_L1", "TT_O2_L2")
    code = {UP: 1, LO: 2, BO: 3, MK: 4, N: 5, W: 6}
    bad = [cp for cp in range(0x110000) if not 0xD800 <= cp <= 0xDFFF
           and _four_bit(l1, l2, cp) != code.get(o200k_class(cp), 0)]
    assert bad == [], bad[:10]


def _two_bit(l1, l2, cp):
    return (l2[l1[cp >> 8] * 64 + ((cp & 255) >> 2)] >> ((cp & 3) * 2)) & 3


def test_base_table_equals_oracle_classes():
    """The GPT-2- and cl100k-style table (letters, numbers, whitespace, other)
    against the oracle's classes for every scalar value: a skew between class
    tables is exactly the failure the paper reports between Unicode versions."""
    from oracle.classes import L, N, W, char_class

    l1, l2 = _arrays("class_table.inc", "TT_CLS_L1", "TT_CLS_L2")
    code = {L: 1, N: 2, W: 3}
    bad = [cp for cp in range(0x110000) if not 0xD800 <= cp <= 0xDFFF
           and _two_bit(l1, l2, cp) != code.get(char_class(cp), 0)]
    assert bad == [], bad[:10]


def test_base_ascii_formula_equals_oracle():
    """The kernels classify ASCII by formula (char_code in tt_tile.hip), not by
    the table: letters, digits, CR/LF and the other whitespace, else other."""
    from oracle.classes import L, N, W, char_class

    def formula(cp):
        if 0 <= (cp | 32) - ord("a") < 26:
            return L
        if 0 <= cp - ord("0") < 10:
            return N
        if cp in (10, 13) or cp == 32 or 0 <= cp - 9 < 5:
            return W
        return None

    for cp in range(128):
        want = char_class(cp)
        assert formula(cp) == (want if want in (L, N, W) else None), cp
