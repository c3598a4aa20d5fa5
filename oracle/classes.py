"""Code-point classes seen by the pre-tokenization patterns (oracle; test infrastructure).

The patterns of both families test three Unicode properties: letters
(``\\p{L}``), numbers (``\\p{N}``) and whitespace (``\\s``).  Every other
code point is "other".  The paper pins these tables by probing the reference
regex engine rather than trusting a library's Unicode version (Sec. 4.1,
table pinning; Sec. 5.2, the Unicode table skew).  ``data/onig_classes.txt``
holds that probe for Oniguruma inside HF tokenizers 0.22.2; it was written by
``data/probe_onig.py``.

The o200k-style pattern also tells upper-case from lower-case letters and
treats combining marks as letter material; ``data/onig_o200k_classes.txt``
holds those sub-classes (Lu|Lt, Ll, Lm|Lo, M), probed from the same engine by
``data/probe_onig_o200k.py``.

The DeepSeek-style pattern also tests punctuation and symbols (``\\p{P}``,
``\\p{S}``); ``data/onig_deepseek_classes.txt`` holds those code points, probed
from the same engine by ``data/probe_onig_deepseek.py``, and its second
splitter names the CJK ideograph, hiragana and katakana ranges directly.

Parity pins: the whole table is compared with a fresh probe of the engine
(tests), and the 25 whitespace code points are checked against the Unicode
White_Space list written out in the test.
"""

import os

L, N, W, O = 1, 2, 3, 0
NAMES = {L: "L", N: "N", W: "W", O: "O"}

_HERE = os.path.dirname(os.path.abspath(__file__))
TABLE_PATH = os.path.join(_HERE, "data", "onig_classes.txt")


def _load():
    table = bytearray(0x110000)  # O everywhere by default
    folds = {}
    code = {"L": L, "N": N, "W": W}
    with open(TABLE_PATH) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "FOLD":
                folds[parts[1]] = frozenset(int(x, 16) for x in parts[2:])
                continue
            a, b, k = int(parts[0], 16), int(parts[1], 16), code[parts[2]]
            for c in range(a, b + 1):
                table[c] = k
    return table, folds


TABLE, FOLDS = _load()


def char_class(cp: int) -> int:
    """Class (L, N, W or O) of one Unicode scalar value."""
    return TABLE[cp]


def classes_of(text: str) -> list:
    """Class of every character of ``text``."""
    t = TABLE
    return [t[ord(c)] for c in text]


def folds_to(ch: str, letter: str) -> bool:
    """True iff ``ch`` matches the ASCII ``letter`` case-insensitively in the engine."""
    return ord(ch) in FOLDS[letter]


# ---- o200k-style sub-classes ---------------------------------------------------
UP, LO, BO, MK = 11, 12, 13, 14  # Lu|Lt, Ll, Lm|Lo, M
O200K_PATH = os.path.join(_HERE, "data", "onig_o200k_classes.txt")


def _load_o200k():
    table = bytearray(0x110000)  # 0: no sub-class
    code = {"UP": UP, "LO": LO, "BO": BO, "MK": MK}
    with open(O200K_PATH) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b, k = line.split()
            for c in range(int(a, 16), int(b, 16) + 1):
                table[c] = code[k]
    return table


O200K_TABLE = _load_o200k()


def o200k_class(cp: int) -> int:
    """UP, LO, BO or MK for letters and marks, else the class of ``char_class`` (N, W or O)."""
    return O200K_TABLE[cp] or TABLE[cp]


def o200k_classes_of(text: str) -> list:
    return [o200k_class(ord(c)) for c in text]


# ---- DeepSeek-style: punctuation and symbols ------------------------------------
DEEPSEEK_PATH = os.path.join(_HERE, "data", "onig_deepseek_classes.txt")


def _load_deepseek():
    table = bytearray(0x110000)  # 1 where \p{P} or \p{S}
    with open(DEEPSEEK_PATH) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b, k = line.split()
            assert k == "PS"
            for c in range(int(a, 16), int(b, 16) + 1):
                table[c] = 1
    return table


PS_TABLE = _load_deepseek()


def is_punct_or_symbol(cp: int) -> bool:
    """\\p{P} or \\p{S} in the engine."""
    return PS_TABLE[cp] != 0


def is_mark(cp: int) -> bool:
    """\\p{M} in the engine."""
    return O200K_TABLE[cp] == MK
