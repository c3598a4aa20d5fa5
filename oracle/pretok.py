"""Leftmost-first regex pre-tokenization, written out by hand (oracle; test infrastructure).

GPT-family pre-tokenizers are a leftmost-first alternation regex with
backtracking; every match starts where the previous one ended (Sec. 1;
Sec. 4.1, "Removing the sequential regex scan").  This module is that
definition and nothing more: at the current position it tries the
alternatives in their order, the first one that matches wins, its match is the
next piece, and the scan continues at the match's end.  Each alternative is
evaluated with the greedy-then-backtrack semantics of its regex operators.
There is no run decomposition here; that reformulation is what the library
implements and what these functions check.

The paper names the pattern lineages but does not print the regexes.  The two
families used here, transcribed from their lineage definitions:

GPT-2 style, alternatives in order
  G1  ``'`` followed by one of ``s t re ve m ll d`` (case-sensitive)
  G2  optional U+0020, then one or more letters           `` ?\\p{L}+``
  G3  optional U+0020, then one or more numbers           `` ?\\p{N}+``
  G4  optional U+0020, then one or more "other" chars     `` ?[^\\s\\p{L}\\p{N}]+``
  G5  whitespace not followed by a non-whitespace char    ``\\s+(?!\\S)``
  G6  whitespace                                          ``\\s+``

cl100k style, alternatives in order
  C1  G1, case-insensitive                                ``(?i:'s|'t|'re|'ve|'m|'ll|'d)``
  C2  one optional char that is not CR/LF, letter or number, then letters
                                                          ``[^\\r\\n\\p{L}\\p{N}]?\\p{L}+``
  C3  one to three numbers                                ``\\p{N}{1,3}``
  C4  optional U+0020, "other" chars, then CR/LF chars    `` ?[^\\s\\p{L}\\p{N}]+[\\r\\n]*``
  C5  whitespace ending in CR/LF                          ``\\s*[\\r\\n]+``
  C6  = G5
  C7  = G6

o200k style, alternatives in order (letters split into upper-case UP = Lu|Lt,
lower-case LO = Ll, "both" BO = Lm|Lo, and marks MK = M, which count as letter
material in the letter sets and as "other" elsewhere; CT is the case-insensitive
contraction suffix of C1, optional here)
  P1  ``[^\\r\\n\\p{L}\\p{N}]?[UP BO MK]*[LO BO MK]+CT?``
  P2  ``[^\\r\\n\\p{L}\\p{N}]?[UP BO MK]+[LO BO MK]*CT?``
  P3  = C3
  P4  optional U+0020, "other" chars, then CR/LF and "/"  `` ?[^\\s\\p{L}\\p{N}]+[\\r\\n/]*``
  P5  = C5,  P6 = G5,  P7 = G6

DeepSeek style (the paper: three splitters applied in sequence, each one
re-splitting every piece of the previous stage, with unmatched stretches kept
as pieces).  Each splitter isolates the leftmost matches of its regex in a
piece, scanning from the piece start; the matches and the stretches between
them are the next stage's pieces, and a regex sees the piece's end as the end
of the text.  The splitters, in order:
  S1  one to three numbers                                ``\\p{N}{1,3}``
  S2  a run of CJK ideographs, hiragana or katakana       ``[\\u4E00-\\u9FA5\\u3040-\\u309F\\u30A0-\\u30FF]+``
  S3  alternatives in order:
      D1  one ASCII punctuation or symbol char, then ASCII letters
                                                          ``[!-/:-@[-`{-~][A-Za-z]+``
      D2  one optional char that is not CR/LF, letter, punctuation or symbol,
          then letters and marks                          ``[^\\r\\n\\p{L}\\p{P}\\p{S}]?[\\p{L}\\p{M}]+``
      D3  optional U+0020, punctuation and symbols, then CR/LF
                                                          `` ?[\\p{P}\\p{S}]+[\\r\\n]*``
      D4  = C5,  D5 = G5,  D6 = G6

Readings taken where the paper is silent: ``\\s`` is the engine's whitespace
class (25 code points), "space" in the optional-space alternatives is U+0020
only, case-insensitive contractions use the engine's case folding (which maps
U+017F to ``s``), and only U+0027 is an apostrophe.
"""

from .classes import (BO, LO, MK, UP, L, N, O, W, classes_of, folds_to, is_mark, is_punct_or_symbol,
                      o200k_classes_of)

GPT2 = "gpt2"
CL100K = "cl100k"
O200K = "o200k"
DEEPSEEK = "deepseek"
PATTERNS = (GPT2, CL100K, O200K, DEEPSEEK)

SUFFIXES = ("s", "t", "re", "ve", "m", "ll", "d")
SP = " "
NL = "\r\n"


def _run(cl, i, k):
    """First index >= i whose class is not k."""
    n = len(cl)
    while i < n and cl[i] == k:
        i += 1
    return i


# -- alternatives: each returns the end of its match at p, or None ----------

def _contraction(text, p, insensitive):
    if text[p] != "'":
        return None
    for suf in SUFFIXES:
        e = p + 1 + len(suf)
        if e > len(text):
            continue
        seg = text[p + 1:e]
        if insensitive:
            ok = all(folds_to(ch, letter) for ch, letter in zip(seg, suf))
        else:
            ok = seg == suf
        if ok:
            return e
    return None


def _opt_space_then_run(text, cl, p, k):
    """`` ?X+`` with X the class k: greedy optional space, backtracking to none."""
    if text[p] == SP:
        e = _run(cl, p + 1, k)
        if e > p + 1:
            return e
    e = _run(cl, p, k)
    return e if e > p else None


def _ws_not_before_nonws(text, cl, p):
    """``\\s+(?!\\S)``: the longest whitespace run, backtracked until the lookahead holds."""
    n = len(text)
    e = _run(cl, p, W)
    for j in range(e, p, -1):
        if j == n or cl[j] == W:
            return j
    return None


def _ws(text, cl, p):
    e = _run(cl, p, W)
    return e if e > p else None


def _gpt2_at(text, cl, p):
    return (_contraction(text, p, False)
            or _opt_space_then_run(text, cl, p, L)
            or _opt_space_then_run(text, cl, p, N)
            or _opt_space_then_run(text, cl, p, O)
            or _ws_not_before_nonws(text, cl, p)
            or _ws(text, cl, p))


def _cl_prefixed_letters(text, cl, p):
    """``[^\\r\\n\\p{L}\\p{N}]?\\p{L}+``"""
    if text[p] not in NL and cl[p] not in (L, N):
        e = _run(cl, p + 1, L)
        if e > p + 1:
            return e
    e = _run(cl, p, L)
    return e if e > p else None


def _cl_numbers(text, cl, p):
    """``\\p{N}{1,3}``"""
    n = len(text)
    e = p
    while e < n and e - p < 3 and cl[e] == N:
        e += 1
    return e if e > p else None


def _cl_other(text, cl, p):
    """`` ?[^\\s\\p{L}\\p{N}]+[\\r\\n]*``"""
    n = len(text)
    starts = (p + 1, p) if text[p] == SP else (p,)
    for s in starts:
        e = _run(cl, s, O)
        if e > s:
            while e < n and text[e] in NL:
                e += 1
            return e
    return None


def _cl_ws_newlines(text, cl, p):
    """``\\s*[\\r\\n]+``: greedy whitespace, backtracked until CR/LF can follow."""
    n = len(text)
    e = _run(cl, p, W)
    for j in range(e, p - 1, -1):
        if j < n and text[j] in NL:
            k = j
            while k < n and text[k] in NL:
                k += 1
            return k
    return None


def _cl100k_at(text, cl, p):
    return (_contraction(text, p, True)
            or _cl_prefixed_letters(text, cl, p)
            or _cl_numbers(text, cl, p)
            or _cl_other(text, cl, p)
            or _cl_ws_newlines(text, cl, p)
            or _ws_not_before_nonws(text, cl, p)
            or _ws(text, cl, p))


# o200k style ---------------------------------------------------------------
_UB = (UP, BO, MK)  # the upper-case letter set [\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]
_LB = (LO, BO, MK)  # the lower-case letter set [\p{Ll}\p{Lm}\p{Lo}\p{M}]


def _run_in(ol, i, ks):
    """First index >= i whose sub-class is not in ks."""
    n = len(ol)
    while i < n and ol[i] in ks:
        i += 1
    return i


def _o200k_suffix(text, e):
    """The optional case-insensitive contraction after a letter body ending at e."""
    if e < len(text):
        c = _contraction(text, e, True)
        if c is not None:
            return c
    return e


def _o200k_letters(text, ol, p, upper_first):
    """P1 (``upper_first`` False): prefix? [UB]* [LB]+ CT?;  P2: prefix? [UB]+ [LB]* CT?.
    The optional prefix is tried first, then the match without it; [UB]* gives
    back characters until [LB]+ can match."""
    n = len(text)
    bodies = []
    if text[p] not in NL and ol[p] in (O, MK, W):  # [^\r\n\p{L}\p{N}]
        bodies.append(p + 1)
    bodies.append(p)
    for b0 in bodies:
        k_end = _run_in(ol, b0, _UB)
        if not upper_first:
            for q in range(k_end, b0 - 1, -1):
                if q < n and ol[q] in _LB:
                    return _o200k_suffix(text, _run_in(ol, q, _LB))
        elif k_end > b0:
            return _o200k_suffix(text, _run_in(ol, k_end, _LB))
    return None


def _o200k_other(text, ol, p):
    """`` ?[^\\s\\p{L}\\p{N}]+[\\r\\n/]*`` (marks are in the set)"""
    n = len(text)
    starts = (p + 1, p) if text[p] == SP else (p,)
    for s in starts:
        e = _run_in(ol, s, (O, MK))
        if e > s:
            while e < n and (text[e] in NL or text[e] == "/"):
                e += 1
            return e
    return None


def _o200k_at(text, cl, ol, p):
    return (_o200k_letters(text, ol, p, False)
            or _o200k_letters(text, ol, p, True)
            or _cl_numbers(text, cl, p)
            or _o200k_other(text, ol, p)
            or _cl_ws_newlines(text, cl, p)
            or _ws_not_before_nonws(text, cl, p)
            or _ws(text, cl, p))


# -- DeepSeek style: three splitters ---------------------------------------------

ASCII_PUNCT = frozenset('!"#$%&\'()*+,-./:;<=>?@[\\]^_`{|}~')
ASCII_LETTERS = frozenset("ABCDEFGHIJKLMNOPQRSTUVWXYZabcdefghijklmnopqrstuvwxyz")


def in_kana_cjk(cp: int) -> bool:
    """The second splitter's set: CJK ideographs U+4E00-9FA5, hiragana U+3040-309F, katakana U+30A0-30FF."""
    return 0x4E00 <= cp <= 0x9FA5 or 0x3040 <= cp <= 0x30FF


def _ds_numbers(text, cl, p, b):
    """S1 ``\\p{N}{1,3}`` at p, inside [p, b)."""
    e = p
    while e < b and e - p < 3 and cl[e] == N:
        e += 1
    return e if e > p else None


def _ds_kana_cjk(text, cl, p, b):
    """S2: a run of the CJK/kana set at p, inside [p, b)."""
    e = p
    while e < b and in_kana_cjk(ord(text[e])):
        e += 1
    return e if e > p else None


def _ds_main(text, cl, p, b):
    """S3 at p, inside [p, b); b is the end of the text for the lookahead."""
    def letter_or_mark(i):
        return cl[i] == L or is_mark(ord(text[i]))

    def ps(i):
        return is_punct_or_symbol(ord(text[i]))

    def run(i, pred):
        while i < b and pred(i):
            i += 1
        return i

    ch = text[p]
    # D1: one ASCII punctuation or symbol char, then ASCII letters
    if ch in ASCII_PUNCT and p + 1 < b and text[p + 1] in ASCII_LETTERS:
        return run(p + 1, lambda i: text[i] in ASCII_LETTERS)
    # D2: the optional prefix first, then without it
    if ch not in NL and cl[p] != L and not ps(p):
        e = run(p + 1, letter_or_mark)
        if e > p + 1:
            return e
    e = run(p, letter_or_mark)
    if e > p:
        return e
    # D3: optional U+0020, punctuation and symbols, then CR/LF
    for st in ((p + 1, p) if ch == SP else (p,)):
        e = run(st, ps)
        if e > st:
            return run(e, lambda i: text[i] in NL)
    # D4-D6: whitespace
    if cl[p] == W:
        e = run(p, lambda i: cl[i] == W)
        for j in range(e - 1, p - 1, -1):  # \s*[\r\n]+ ends after the last CR/LF of the run
            if text[j] in NL:
                return j + 1
        for j in range(e, p, -1):  # \s+(?!\S)
            if j == b or cl[j] == W:
                return j
        return e  # \s+
    return None


def _isolated(text, cl, spans, match_at):
    """One splitter with the Isolated behaviour over each span: the leftmost
    matches, scanning from the span start, and the stretches between them."""
    out = []
    for a, b in spans:
        p = gap = a
        while p < b:
            e = match_at(text, cl, p, b)
            if e is None:
                p += 1
                continue
            if gap < p:
                out.append((gap, p))
            out.append((p, e))
            p = gap = e
        if gap < b:
            out.append((gap, b))
    return out


def _deepseek(text, cl):
    spans = [(0, len(text))] if text else []
    for match_at in (_ds_numbers, _ds_kana_cjk, _ds_main):
        spans = _isolated(text, cl, spans, match_at)
    return spans


def pretokenize(text: str, pattern: str) -> list:
    """Pieces of ``text`` as (start, end) character spans, in order, tiling the text."""
    cl = classes_of(text)
    if pattern == DEEPSEEK:
        return _deepseek(text, cl)
    if pattern == GPT2:
        step = _gpt2_at
    elif pattern == CL100K:
        step = _cl100k_at
    elif pattern == O200K:
        ol = o200k_classes_of(text)

        def step(t, c, p):
            return _o200k_at(t, c, ol, p)
    else:
        raise ValueError("unknown pattern %r" % (pattern,))
    spans = []
    p = 0
    n = len(text)
    while p < n:
        e = step(text, cl, p)
        assert e is not None and e > p, "no alternative matched at %d" % p
        spans.append((p, e))
        p = e
    return spans


def pieces(text: str, pattern: str) -> list:
    """Pieces of ``text`` as strings."""
    return [text[a:b] for a, b in pretokenize(text, pattern)]


def piece_byte_starts(text: str, pattern: str) -> list:
    """UTF-8 byte offset of the first byte of every piece."""
    starts = []
    off = 0
    for a, b in pretokenize(text, pattern):
        starts.append(off)
        off += len(text[a:b].encode("utf-8"))
    return starts
