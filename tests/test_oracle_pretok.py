"""Pins of the oracle's pre-tokenizer (CPU only).

The oracle's matcher is checked against things other than itself:
  * worked examples produced by the reference regex engine (tests/golden);
  * a second matcher: a generic backtracking regex interpreter run on ASTs
    transcribed from the pattern text, by brute force over every string of
    up to five characters from a 13-character alphabet;
  * the Oniguruma engine itself (HF tokenizers 0.22.2, the engine the paper
    pins) on random strings and on the seeded texts;
  * the tiling invariant: the pieces concatenate to the input.
"""

import itertools
import os
import random

import pytest

from oracle.pretok import pretokenize, pieces
from regex_interp import split as interp_split

HERE = os.path.dirname(os.path.abspath(__file__))
PATTERNS = ("gpt2", "cl100k", "o200k")

REGEX = {
    "gpt2": r"'s|'t|'re|'ve|'m|'ll|'d| ?\p{L}+| ?\p{N}+| ?[^\s\p{L}\p{N}]+|\s+(?!\S)|\s+",
    "cl100k": r"(?i:'s|'t|'re|'ve|'m|'ll|'d)|[^\r\n\p{L}\p{N}]?\p{L}+|\p{N}{1,3}| ?[^\s\p{L}\p{N}]+[\r\n]*"
              r"|\s*[\r\n]+|\s+(?!\S)|\s+",
    "o200k": r"[^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]*[\p{Ll}\p{Lm}\p{Lo}\p{M}]+(?i:'s|'t|'re|'ve|'m|'ll|'d)?"
             r"|[^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]+[\p{Ll}\p{Lm}\p{Lo}\p{M}]*(?i:'s|'t|'re|'ve|'m|'ll|'d)?"
             r"|\p{N}{1,3}| ?[^\s\p{L}\p{N}]+[\r\n/]*|\s*[\r\n]+|\s+(?!\S)|\s+",
}


def _unescape(s):
    s = s.replace("\\s", " ").replace("\\xa0", " ").replace("\\'", "'")
    return s.encode("latin-1", "backslashreplace").decode("unicode_escape") if "\\" in s else s


def _golden():
    rows = []
    with open(os.path.join(HERE, "golden", "pretok_examples.txt"), encoding="utf-8") as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            src, g2, cl = line.rstrip("\n").split("\t")
            rows.append((_unescape(src), [_unescape(p) for p in g2.split(" | ")],
                         [_unescape(p) for p in cl.split(" | ")]))
    return rows


@pytest.mark.parametrize("row", _golden(), ids=lambda r: repr(r[0]))
def test_worked_examples(row):
    src, g2, cl = row
    assert pieces(src, "gpt2") == g2
    assert pieces(src, "cl100k") == cl


ALPHA13 = list("asl'S1 \n\t.re\r")
# o200k: upper, lower, title-case (Lt), other letter (Lo), modifier letter (Lm),
# combining mark, and the characters its other alternatives single out
ALPHA_O200K = list("aS1 \n\t'./\r") + ["ǅ", "中", "ʰ", "\u0301"]


def _golden_o200k():
    rows = []
    with open(os.path.join(HERE, "golden", "pretok_o200k_examples.txt"), encoding="utf-8") as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            src, pcs = line.rstrip("\n").split("\t")
            rows.append((_unescape(src), [_unescape(p) for p in pcs.split(" | ")]))
    return rows


@pytest.mark.parametrize("row", _golden_o200k(), ids=lambda r: repr(r[0]))
def test_worked_examples_o200k(row):
    src, want = row
    assert pieces(src, "o200k") == want


@pytest.mark.parametrize("pattern", PATTERNS)
def test_brute_force_against_backtracking_interpreter(pattern):
    alpha = ALPHA_O200K if pattern == "o200k" else ALPHA13
    n = 0
    for length in range(1, 5):
        for tup in itertools.product(alpha, repeat=length):
            s = "".join(tup)
            assert pretokenize(s, pattern) == interp_split(s, pattern), repr(s)
            n += 1
    assert n == sum(len(alpha) ** k for k in range(1, 5))


WIDE = list("asS1 \n\t'.\r") + ["\u0085", " ", "ſ", "²", "中", "。", "\U0001f600",
                                 "́", "　", "½", "А", "t", "T", "d", "D", "m", "M",
                                 "l", "L", "v", "V", "e", "E", "R", "_", "-", " ", "\x1c", "/", "ǅ", "ʰ",
                                 "É", "ä", "\u0308", "Ж"]


@pytest.mark.parametrize("pattern", PATTERNS)
def test_random_against_backtracking_interpreter(pattern):
    rng = random.Random(7 + len(pattern))
    for _ in range(3000):
        s = "".join(rng.choice(WIDE) for _ in range(rng.randint(1, 14)))
        assert pretokenize(s, pattern) == interp_split(s, pattern), repr(s)


def _onig(pattern):
    tk = pytest.importorskip("tokenizers")
    sp = tk.pre_tokenizers.Split(tk.Regex(REGEX[pattern]), behavior="isolated")
    return lambda s: [o for _, o in sp.pre_tokenize_str(s)]


@pytest.mark.parametrize("pattern", PATTERNS)
def test_random_against_oniguruma(pattern):
    onig = _onig(pattern)
    rng = random.Random(99 + len(pattern))
    for _ in range(20000):
        s = "".join(rng.choice(WIDE) for _ in range(rng.randint(1, 16)))
        assert pretokenize(s, pattern) == onig(s), repr(s)


def test_worked_examples_o200k_against_oniguruma():
    onig = _onig("o200k")
    for src, want in _golden_o200k():
        assert [src[a:b] for a, b in onig(src)] == want, repr(src)


@pytest.mark.parametrize("k", [1, 2, 4])
def test_seeded_text_against_oniguruma(k):
    from conftest import config_bytes, pattern_of

    pattern = pattern_of(k)
    onig = _onig(pattern)
    text = config_bytes(k).decode("utf-8")[:200_000]
    assert pretokenize(text, pattern) == onig(text)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_pieces_tile_the_text(k):
    from conftest import config_bytes, pattern_of

    text = config_bytes(k).decode("utf-8")
    spans = pretokenize(text, pattern_of(k))
    assert spans[0][0] == 0 and spans[-1][1] == len(text)
    assert all(a < b for a, b in spans)
    assert all(spans[i][1] == spans[i + 1][0] for i in range(len(spans) - 1))
    assert "".join(text[a:b] for a, b in spans) == text


def test_planted_fault_is_caught():
    """Harness validation: a pre-tokenizer with one rule dropped disagrees with the interpreter."""
    import oracle.pretok as P

    orig = P._cl_numbers

    def wrong(text, cl, p):  # digit runs without the chunks of three
        e = p
        while e < len(text) and cl[e] == P.N:
            e += 1
        return e if e > p else None

    P._cl_numbers = wrong
    try:
        assert P.pretokenize("12345", "cl100k") != interp_split("12345", "cl100k")
    finally:
        P._cl_numbers = orig
