"""Right-context piece starts of the walked patterns, pinned to the oracle.

Besides the synchronizing pairs (``test_repair_host.py``), the tile kernel's
walks for the o200k- and DeepSeek-style patterns start segments at two kinds
of whitespace that begin a piece whatever text lies to their left, given the
text to their right (Section 4.1's alternatives):

  A. one-byte whitespace (not CR/LF) followed by a character that is not
     whitespace (DeepSeek-style: and neither a number nor a CJK/kana
     character, which end the third splitter's stretch);
  B. whitespace (not CR/LF) right after CR/LF whose whitespace run holds no
     further CR/LF.

The rules are restated here from their definitions and checked with the
oracle's pre-tokenizer as judge, exhaustively over short strings of a
class-representative alphabet (every left context up to that length) and on
seeded random strings.  A weakened rule must fail the same check.
"""

import itertools
import random

import pytest

from oracle.classes import N, W, char_class
from oracle.pretok import in_kana_cjk, pretokenize

ALPHA = {
    # U+0020, tab, LF, CR, U+3000 (multi-byte whitespace), lower and upper
    # letters, a digit, symbols (apostrophe, "/", "}"), a Lo letter and a mark
    "o200k": [" ", "\t", "\n", "\r", "　", "a", "S", "1", "'", "/", "}", "中", "́"],
    # U+0020, tab, LF, CR, U+3000, a letter, a digit, ASCII punctuation, a
    # CJK ideograph, a mark, a control character
    "deepseek": [" ", "\t", "\n", "\r", "　", "a", "1", ".", "中", "́", "\x01"],
}
MAX_LEN = {"o200k": 5, "deepseek": 5}


def _ws(ch):
    return char_class(ord(ch)) == W and ch not in "\r\n"


def walk_starts(text, pattern, weaken=None):
    """Character positions of rules A and B (``weaken`` drops one condition,
    for the negative test)."""
    out = set()
    n = len(text)
    for i, ch in enumerate(text):
        if not _ws(ch):
            continue
        if len(ch.encode("utf-8")) == 1 and i + 1 < n:
            nx = text[i + 1]
            solid = char_class(ord(nx)) != W
            if pattern == "deepseek" and weaken != "stretch":
                solid = solid and char_class(ord(nx)) != N and not in_kana_cjk(ord(nx))
            if solid:
                out.add(i)
        if i >= 1 and text[i - 1] in "\r\n":
            j = i
            while j < n and _ws(text[j]):
                j += 1
            if weaken == "crlf" or j == n or text[j] not in "\r\n":
                out.add(i)
    return out


def _violations(text, pattern, weaken=None):
    starts = {a for a, _ in pretokenize(text, pattern)}
    return sorted(walk_starts(text, pattern, weaken) - starts)


@pytest.mark.parametrize("pattern", ["o200k", "deepseek"])
def test_walk_starts_exhaustive_short_strings(pattern):
    hits = 0
    for n in range(2, MAX_LEN[pattern] + 1):
        for tup in itertools.product(ALPHA[pattern], repeat=n):
            text = "".join(tup)
            bad = _violations(text, pattern)
            assert not bad, "%s: %r: no piece start at %s" % (pattern, text, bad)
            hits += len(walk_starts(text, pattern))
    assert hits > 20000


@pytest.mark.parametrize("pattern", ["o200k", "deepseek"])
def test_walk_starts_random_strings(pattern):
    rng = random.Random(0xB0B + len(pattern))
    alphabet = ALPHA[pattern] + ["  ", "\n    ", "\r\n  ", "  \n", "x", "A", " ", "ʰ", "23", "-", '"']
    hits = 0
    for _ in range(3000):
        text = "".join(rng.choice(alphabet) for _ in range(rng.randint(4, 30)))
        bad = _violations(text, pattern)
        assert not bad, "%s: %r: no piece start at %s" % (pattern, text, bad)
        hits += len(walk_starts(text, pattern))
    assert hits > 3000


@pytest.mark.parametrize("pattern,weaken,text", [
    ("o200k", "crlf", "\n \n"),         # the CR/LF alternative runs on to the later LF
    ("deepseek", "crlf", "\n\t\r\n"),
    ("deepseek", "stretch", "a  1"),    # the stretch ends at the number: "\s+(?!\S)" takes both spaces
    ("deepseek", "stretch", "a  中"),
])
def test_weakened_rules_fail(pattern, weaken, text):
    assert _violations(text, pattern) == []
    assert _violations(text, pattern, weaken) != []
