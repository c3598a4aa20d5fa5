"""Incremental repair, host side, without a GPU.

The library's splice check rests on one property of the pre-tokenizer: at a
synchronizing boundary p (a class transition from the pattern's set), every
text has a piece boundary, the pieces right of p do not depend on the text
before p's left neighbour, and the pieces left of p do not depend on the text
after p's right neighbour (Appendix, Definition d:cert and "Discharging the
certificate per family").  These tests pin the library's sets
(``tt_sync_boundaries``) to that property with the oracle's pre-tokenizer as
judge: exhaustively over short strings of a class-representative alphabet and
on seeded random strings.  They then feed the library's splice decision
(``tt_splice_plan``) with records computed by the oracle and check that every
admitted splice reproduces the oracle's tokenization of the whole text.
"""

import itertools
import random

import pytest

from conftest import oracle_table
from oracle.pretok import pretokenize
from oracle.spans import encode_with_spans
from paper_2607_29678_amd import splice_plan, sync_boundaries

# one character of every class and identity the rules distinguish
ALPHA = {
    "gpt2": list("as1 \n\t'.rel") + ["\r"],
    "cl100k": list("aS1 \n\t'.rl") + ["\r", "ſ", " "],
    # upper, lower, Lo, Lm, a mark, "/" (absorbed after CR/LF by symbol pieces)
    "o200k": list("aS1 \n\t'./") + ["\u4e2d", "\u02b0", "\u0301", "\r"],
    # ASCII and other letters, a mark, a number, ASCII and other punctuation,
    # U+0020, tab, LF, a control char, and letter, mark, symbol and unassigned
    # code point of the CJK/kana ranges
    "deepseek": list("a1. \t\n\x01") + ["\u00e9", "\u0301", "\u3002", "\u4e2d", "\u3099", "\u309b", "\u3040"],
}
MAX_LEN = {"gpt2": 5, "cl100k": 5, "o200k": 5, "deepseek": 4}
EXTRA = ["中", "。", "²", "\U0001f600", "́", "　", "\u0085", "А", "\u00c9", "\u01c5", "\u02b0", "/", "T", "D"]


def _starts(text, pattern, memo):
    r = memo.get(text)
    if r is None:
        r = memo[text] = frozenset(a for a, _ in pretokenize(text, pattern))
    return r


def certificate_violation(text, p, pattern, memo):
    """None if character position p of `text` is a splice certificate for every
    split of the text around it, else a description of the first failure."""
    n = len(text)
    full = _starts(text, pattern, memo)
    if p not in full:
        return "no piece boundary at %d" % p
    left = {a for a in full if a < p}
    right = {a for a in full if a >= p}
    for m in range(p + 1, n):  # the stored text A = text[:m] (ends after p)
        sm = _starts(text[:m], pattern, memo)
        if p not in sm or {a for a in sm if a < p} != left:
            return "prefix of %d characters changes the pieces left of %d" % (m, p)
    for x in range(0, p):  # a window starting at x <= p - 1
        sx = _starts(text[x:], pattern, memo)
        if {a + x for a in sx if a + x >= p} != right:
            return "window from %d changes the pieces right of %d" % (x, p)
    return None


def _char_positions(text):
    """byte offset -> character index for character starts."""
    out, off = {}, 0
    for i, ch in enumerate(text):
        out[off] = i
        off += len(ch.encode("utf-8"))
    return out


def _check_string(text, pattern, memo):
    data = text.encode("utf-8")
    mask = sync_boundaries(data, pattern)
    cpos = _char_positions(text)
    hits = 0
    for b in range(1, len(data)):
        if not mask[b]:
            continue
        assert b in cpos, "boundary inside a character: %r at byte %d" % (text, b)
        why = certificate_violation(text, cpos[b], pattern, memo)
        assert why is None, "%s: %r at character %d: %s" % (pattern, text, cpos[b], why)
        hits += 1
    return hits


@pytest.mark.parametrize("pattern", ["gpt2", "cl100k", "o200k", "deepseek"])
def test_sync_boundaries_exhaustive_short_strings(pattern):
    """Every string of up to 5 characters over the alphabet (4 for the
    DeepSeek-style alphabet of 14): each position the library calls
    synchronizing is a certificate for every split."""
    memo = {}
    hits = 0
    for n in range(2, MAX_LEN[pattern] + 1):
        for tup in itertools.product(ALPHA[pattern], repeat=n):
            hits += _check_string("".join(tup), pattern, memo)
    assert hits > 10000  # the sets are not empty


@pytest.mark.parametrize("pattern", ["gpt2", "cl100k", "o200k", "deepseek"])
def test_sync_boundaries_random_strings(pattern):
    rng = random.Random(0x5A11 + len(pattern))
    alphabet = ALPHA[pattern] + EXTRA + ["a"] * 6 + ["1"] * 4 + [" "] * 4
    memo = {}
    hits = 0
    for _ in range(1500):
        text = "".join(rng.choice(alphabet) for _ in range(rng.randint(6, 18)))
        hits += _check_string(text, pattern, memo)
    assert hits > 1000


def test_certificate_checker_catches_unsafe_transitions():
    """The checker itself: transitions left out of the sets on purpose fail it."""
    memo = {}
    # GPT-2: a letter after U+0020 joins it (" b" is one piece)
    assert certificate_violation("a b", 2, "gpt2", memo) is not None
    # GPT-2: a contraction suffix after an apostrophe
    assert certificate_violation("x's", 2, "gpt2", memo) is not None
    # cl100k: a letter after a tab takes the tab as its prefix
    assert certificate_violation("a\tb", 2, "cl100k", memo) is not None
    # cl100k: a lone symbol prefixes the letters after it, unless U+0020 precedes it
    assert certificate_violation("a.b", 2, "cl100k", memo) is not None
    # cl100k: digit groups count from the head of the number run
    assert certificate_violation("12345", 3, "cl100k", memo) is not None
    # cl100k: a symbol piece absorbs the CR/LF after it
    assert certificate_violation("a.\nb", 2, "cl100k", memo) is not None
    # o200k: an upper-case run is split after its last Lo/Lm letter only if no
    # lower-case letter follows the run ("中A." splits at 1, "中Ab" does not)
    assert certificate_violation("\u4e2dAb", 1, "o200k", memo) is not None
    # o200k: a symbol piece absorbs CR/LF and "/" after it
    assert certificate_violation("x.\n/y", 3, "o200k", memo) is not None
    # o200k: a mark extends the letters before it
    assert certificate_violation("a\u0301b", 1, "o200k", memo) is not None
    # DeepSeek: ASCII punctuation takes the ASCII letters after it
    assert certificate_violation("x.ab", 2, "deepseek", memo) is not None
    # DeepSeek: a punctuation run takes the CR/LF after it
    assert certificate_violation("a.\nb", 2, "deepseek", memo) is not None
    # and safe ones pass
    assert certificate_violation(".\u00e9", 1, "deepseek", memo) is None
    assert certificate_violation("ab.c", 2, "cl100k", memo) is None
    assert certificate_violation("abCd", 2, "o200k", memo) is None


def test_sync_boundaries_reject_invalid_neighbours():
    assert list(sync_boundaries(b"a\xff1", "gpt2")) == [0, 0, 0]
    assert list(sync_boundaries(b"", "gpt2")) == []
    # a multi-byte letter before a digit: the boundary is the digit's first byte
    m = sync_boundaries("é1".encode(), "cl100k")
    assert list(m) == [0, 0, 1]


# ---- the splice decision on oracle records ----------------------------------

def _window_start(data: bytes, a_len: int, w: int) -> int:
    x, c = a_len, 0
    while x > 0 and c < w:
        x -= 1
        c += (data[x] & 0xC0) != 0x80
    return x


def _max_token_bytes(table):
    return max(len(v) for v in table.vocab)


def _plan_case(a: bytes, b: bytes, table, pattern, w):
    """Returns None if rejected, else asserts the splice equals the oracle and returns True."""
    text = a + b
    x = _window_start(text, len(a), w)
    if x == 0:
        return None
    c_ids, c_spans = encode_with_spans(a, table, pattern)
    f_ids, f_spans = encode_with_spans(text[x:], table, pattern)
    chars_before = len(text[:x].decode("utf-8"))
    f_spans = [(p + x, q + x, c + chars_before, d + chars_before) for p, q, c, d in f_spans]
    plan = splice_plan(text, len(a), x, c_ids, c_spans, f_ids, f_spans, _max_token_bytes(table), pattern)
    if plan is None:
        return None
    kc, ff = plan
    want_ids, want_spans = encode_with_spans(text, table, pattern)
    got_ids = list(c_ids[:kc]) + list(f_ids[ff:])
    got_spans = [tuple(s) for s in c_spans[:kc]] + [tuple(s) for s in f_spans[ff:]]
    assert got_ids == want_ids, (a[-40:], b[:40])
    assert got_spans == [tuple(s) for s in want_spans]
    return True


@pytest.mark.parametrize("k,pattern", [(1, "gpt2"), (4, "cl100k")])
def test_splice_plan_on_seeded_text(k, pattern):
    """Cut seeded text at random characters: every admitted splice is exact,
    and on natural text the first window is almost always admitted."""
    from workloads import textgen

    table = oracle_table(k)
    text = textgen.config_text(k)[:6000]
    rng = random.Random(77 + k)
    accepted = 0
    trials = 60
    for _ in range(trials):
        cut = rng.randint(300, len(text) - 200)
        end = min(len(text), cut + rng.randint(1, 150))
        a = text[:cut].encode("utf-8")
        b = text[cut:end].encode("utf-8")
        if _plan_case(a, b, table, pattern, 128):
            accepted += 1
    assert accepted >= trials * 0.9, accepted


ADVERSARIAL = [
    # digit grouping: appended digits regroup the whole number run (cl100k)
    ("x " + "1" * 400, "1"),
    ("y " + "12" * 200, "345"),
    # whitespace lookahead and newline absorption
    ("abc" + " " * 300, "d"),
    ("q." + "\n" * 300, "\n z"),
    ("r" + "\r\n" * 200, " s"),
    # a contraction completed by the append
    ("text " * 60 + "don", "'t"),
    # an append that joins the last piece
    ("lorem ipsum " * 30 + " pipe", "line"),
]


@pytest.mark.parametrize("pattern,k", [("gpt2", 1), ("cl100k", 4)])
def test_splice_plan_adversarial(pattern, k):
    """Appends built to move boundaries far back: whatever the decision, an
    admitted splice is exact (long same-class runs leave no certificate in a
    narrow window, so those windows are rejected)."""
    table = oracle_table(k)
    for a, b in ADVERSARIAL:
        for w in (16, 64, 128, 1024):
            _plan_case(a.encode(), b.encode(), table, pattern, w)
    # a 400-digit run with a 64-character window has no synchronizing boundary
    assert _plan_case(("x " + "1" * 400).encode(), b"1", table, "cl100k", 64) is None


def test_splice_plan_argument_errors():
    from paper_2607_29678_amd import TokTierError

    with pytest.raises(TokTierError):
        splice_plan(b"abc", 2, 0, [1], [(0, 1, 0, 1)], [1], [(0, 1, 0, 1)], 4)  # x must be > 0
    with pytest.raises(TokTierError):
        splice_plan(b"abc", 5, 1, [1], [(0, 1, 0, 1)], [1], [(0, 1, 0, 1)], 4)  # A longer than the text


def test_deepseek_sync_boundaries_long_contexts():
    """The DeepSeek-style set on longer strings (24 to 64 characters) than the
    exhaustive and random checks above, so that every listed transition is met
    with long runs on both sides (letter runs, punctuation runs absorbing CR/LF,
    whitespace runs with and without CR/LF, number groups, CJK/kana stretches,
    unmatched stretches of control characters)."""
    rng = random.Random(0xD5EE)
    runs = ["abc", "Zq", "été", "́", "...", "、。", "¿", "   ", "\t \t", "\r\n", "\n\n ",
            "\x01\x02", "12345", "中文", "゙", "゛゛", "぀", "'s", " .", "-x"]
    memo = {}
    hits = 0
    for _ in range(1000):
        text = ""
        target = rng.randint(24, 64)
        while len(text) < target:
            text += rng.choice(runs)
        hits += _check_string(text, "deepseek", memo)
    assert hits > 10000
