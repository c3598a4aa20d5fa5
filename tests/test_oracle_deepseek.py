"""Pins of the oracle's DeepSeek-style pre-tokenizer (CPU only).

The DeepSeek-style front end is three splitters applied in sequence, each one
re-splitting every piece of the stage before and keeping unmatched stretches
as pieces (Sec. 4.1).  The oracle writes the three matchers out by hand and
composes them; it is checked against:
  * worked examples (tests/golden/pretok_deepseek_examples.txt), each also
    checked against the engine;
  * the engine's own composition: HF tokenizers 0.22.2 (Oniguruma, the engine
    the paper pins), a Sequence of three Split pre-tokenizers with the
    Isolated behaviour, on every string of up to four characters over a
    16-character alphabet, on random strings over a wide alphabet and on the
    multilingual seeded text;
  * the tiling invariant;
  * the punctuation-and-symbol table: its file is SHA-256 pinned and equals a
    fresh probe of the engine (slow).
"""

import hashlib
import itertools
import os
import random

import pytest

from oracle.pretok import pieces, pretokenize

HERE = os.path.dirname(os.path.abspath(__file__))

# the three splitters of the DeepSeek-V3 lineage's pre-tokenizer
SPLITTERS = (
    r"\p{N}{1,3}",
    "[一-龥぀-ゟ゠-ヿ]+",
    r"[!" + '"' + r"#$%&'()*+,\-./:;<=>?@\[\\\]^_`{|}~][A-Za-z]+|[^\r\n\p{L}\p{P}\p{S}]?[\p{L}\p{M}]+"
    r"| ?[\p{P}\p{S}]+[\r\n]*|\s*[\r\n]+|\s+(?!\S)|\s+",
)


def _engine():
    tk = pytest.importorskip("tokenizers")
    seq = tk.pre_tokenizers.Sequence([tk.pre_tokenizers.Split(tk.Regex(r), behavior="isolated")
                                      for r in SPLITTERS])
    return lambda s: [o for _, o in seq.pre_tokenize_str(s)]


def _unescape(s):
    s = s.replace("\\s", " ").replace("\\'", "'")
    return s.encode("latin-1", "backslashreplace").decode("unicode_escape") if "\\" in s else s


def _golden():
    rows = []
    with open(os.path.join(HERE, "golden", "pretok_deepseek_examples.txt"), encoding="utf-8") as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            src, pcs = line.rstrip("\n").split("\t")
            rows.append((_unescape(src), [_unescape(p) for p in pcs.split(" | ")]))
    return rows


@pytest.mark.parametrize("row", _golden(), ids=lambda r: repr(r[0]))
def test_worked_examples(row):
    src, want = row
    assert pieces(src, "deepseek") == want


def test_worked_examples_against_the_engine():
    eng = _engine()
    for src, want in _golden():
        assert [src[a:b] for a, b in eng(src)] == want, repr(src)


# one character of every class the splitters tell apart: ASCII letters, a
# non-ASCII letter, a mark, numbers (ASCII and not), CR, LF, tab, U+0020,
# ASCII punctuation (one of which starts D1), a non-ASCII symbol, a CJK
# ideograph, a kana symbol inside the second splitter's range, a control char
ALPHA = list("aZ1 \n\r\t.'") + ["é", "́", "²", "中", "゛", "😀", "\x01"]


def test_brute_force_against_the_engine():
    eng = _engine()
    n = 0
    for length in range(1, 5):
        for tup in itertools.product(ALPHA, repeat=length):
            s = "".join(tup)
            assert pretokenize(s, "deepseek") == eng(s), repr(s)
            n += 1
    assert n == sum(len(ALPHA) ** k for k in range(1, 5))


WIDE = list("azAZ019 \n\r\t.,!$(_`~-'/") + [
    " ", "\u0085", "　", "é", "Ж", "ǅ", "ʰ", "́", "̈", "²", "¼", "Ⅳ", "中", "文", "。", "，",
    "あ", "カ", "゛", "゙", "・", "ー", "゠", "\U0001f600", "€", "\x01", "\x1c", "​", "͸", "ſ"]


def test_random_against_the_engine():
    eng = _engine()
    rng = random.Random(0xD5)
    for _ in range(20000):
        s = "".join(rng.choice(WIDE) for _ in range(rng.randint(1, 18)))
        assert pretokenize(s, "deepseek") == eng(s), repr(s)


def test_seeded_text_against_the_engine():
    from conftest import config_bytes

    text = config_bytes(4).decode("utf-8")[:200_000]
    spans = pretokenize(text, "deepseek")
    assert spans == _engine()(text)
    assert spans[0][0] == 0 and spans[-1][1] == len(text)
    assert all(spans[i][1] == spans[i + 1][0] and spans[i][0] < spans[i][1] for i in range(len(spans) - 1))


def test_pieces_tile_the_text():
    from conftest import config_bytes

    for k in (1, 3, 4):
        text = config_bytes(k).decode("utf-8")[:300_000]
        assert "".join(pieces(text, "deepseek")) == text


def test_planted_fault_is_caught():
    """Harness validation: the oracle with D1 switched off disagrees with the engine."""
    import oracle.pretok as P

    orig = P.ASCII_LETTERS
    P.ASCII_LETTERS = frozenset()  # D1 never matches
    try:
        assert P.pretokenize(".abc", "deepseek") != _engine()(".abc")
    finally:
        P.ASCII_LETTERS = orig
    assert pretokenize(".abc", "deepseek") == _engine()(".abc")


def test_class_table_file_pinned():
    from oracle.classes import DEEPSEEK_PATH

    with open(DEEPSEEK_PATH, "rb") as f:
        assert hashlib.sha256(f.read()).hexdigest() == \
            "a2f66ad8bfd39db625744b365d5ea3e20f7cb42035755fedf8e78a6c2445903b"


@pytest.mark.slow
def test_class_table_equals_fresh_engine_probe():
    tk = pytest.importorskip("tokenizers")
    from oracle.classes import PS_TABLE

    cps = [c for c in range(0x110000) if not 0xD800 <= c <= 0xDFFF]
    text = "".join(map(chr, cps))
    sp = tk.pre_tokenizers.Split(tk.Regex(r"[\p{P}\p{S}]"), behavior="removed")
    left = bytearray(len(cps))
    for _, (a, b) in sp.pre_tokenize_str(text):
        left[a:b] = b"\x01" * (b - a)
    assert {cps[i] for i in range(len(cps)) if not left[i]} == {c for c in range(0x110000) if PS_TABLE[c]}
