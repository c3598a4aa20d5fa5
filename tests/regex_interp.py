"""A tiny backtracking regex interpreter, used only by tests as a second matcher.

It knows nothing about run rules or about the oracle's hand-written
alternatives: it interprets a pattern AST (alternation, sequence, character
class, greedy bounded repetition, negative lookahead, case-insensitive
literal) with ordinary backtracking, and pre-tokenizes by repeated
leftmost-first matching.  The pattern ASTs below are transcriptions of the
regex text of the two pattern families.
"""

from oracle.classes import BO, LO, MK, UP, char_class, folds_to, o200k_class, L, N, W


class Node:
    pass


class Alt(Node):
    def __init__(self, *opts):
        self.opts = opts


class Seq(Node):
    def __init__(self, *items):
        self.items = items


class Cls(Node):
    def __init__(self, pred):
        self.pred = pred


class Rep(Node):
    def __init__(self, node, lo, hi):
        self.node, self.lo, self.hi = node, lo, hi


class NotAhead(Node):
    def __init__(self, node):
        self.node = node


def lit(s, ci=False):
    if ci:
        return Seq(*[Cls(lambda c, ch=ch: (c == "'" if ch == "'" else folds_to(c, ch))) for ch in s])
    return Seq(*[Cls(lambda c, ch=ch: c == ch) for ch in s])


INF = 1 << 30


def match(node, text, pos, k):
    """Continuation-passing backtracking matcher: calls k(end) for each way to match, first success wins."""
    if isinstance(node, Cls):
        if pos < len(text) and node.pred(text[pos]):
            return k(pos + 1)
        return None
    if isinstance(node, Seq):
        def go(i, p):
            if i == len(node.items):
                return k(p)
            return match(node.items[i], text, p, lambda q: go(i + 1, q))
        return go(0, pos)
    if isinstance(node, Alt):
        for o in node.opts:
            r = match(o, text, pos, k)
            if r is not None:
                return r
        return None
    if isinstance(node, Rep):
        def rep(count, p):
            if count < node.hi:  # greedy: try one more first
                r = match(node.node, text, p, lambda q: rep(count + 1, q) if q > p else None)
                if r is not None:
                    return r
            if count >= node.lo:
                return k(p)
            return None
        return rep(0, pos)
    if isinstance(node, NotAhead):
        if match(node.node, text, pos, lambda q: q) is not None:
            return None
        return k(pos)
    raise TypeError(node)


def is_L(c):
    return char_class(ord(c)) == L


def is_N(c):
    return char_class(ord(c)) == N


def is_s(c):
    return char_class(ord(c)) == W


SP = Cls(lambda c: c == " ")
LET = Cls(is_L)
NUM = Cls(is_N)
OTHER = Cls(lambda c: not (is_s(c) or is_L(c) or is_N(c)))
WS = Cls(is_s)
NONWS = Cls(lambda c: not is_s(c))
CRLF = Cls(lambda c: c in "\r\n")
NOT_CRLF_L_N = Cls(lambda c: c not in "\r\n" and not is_L(c) and not is_N(c))


def opt(n):
    return Rep(n, 0, 1)


def plus(n):
    return Rep(n, 1, INF)


def star(n):
    return Rep(n, 0, INF)


CONTRACTIONS = ["'s", "'t", "'re", "'ve", "'m", "'ll", "'d"]

# 's|'t|'re|'ve|'m|'ll|'d| ?\p{L}+| ?\p{N}+| ?[^\s\p{L}\p{N}]+|\s+(?!\S)|\s+
GPT2 = Alt(*[lit(c) for c in CONTRACTIONS],
           Seq(opt(SP), plus(LET)),
           Seq(opt(SP), plus(NUM)),
           Seq(opt(SP), plus(OTHER)),
           Seq(plus(WS), NotAhead(NONWS)),
           plus(WS))

# (?i:'s|'t|'re|'ve|'m|'ll|'d)|[^\r\n\p{L}\p{N}]?\p{L}+|\p{N}{1,3}| ?[^\s\p{L}\p{N}]+[\r\n]*|\s*[\r\n]+|\s+(?!\S)|\s+
CL100K = Alt(Alt(*[lit(c, ci=True) for c in CONTRACTIONS]),
             Seq(opt(NOT_CRLF_L_N), plus(LET)),
             Rep(NUM, 1, 3),
             Seq(opt(SP), plus(OTHER), star(CRLF)),
             Seq(star(WS), plus(CRLF)),
             Seq(plus(WS), NotAhead(NONWS)),
             plus(WS))

UB = Cls(lambda c: o200k_class(ord(c)) in (UP, BO, MK))  # [\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]
LB = Cls(lambda c: o200k_class(ord(c)) in (LO, BO, MK))  # [\p{Ll}\p{Lm}\p{Lo}\p{M}]
CRLF_SLASH = Cls(lambda c: c in "\r\n/")
CONTRACTION = Alt(*[lit(c, ci=True) for c in CONTRACTIONS])

# [^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]*[\p{Ll}\p{Lm}\p{Lo}\p{M}]+(?i:'s|'t|'re|'ve|'m|'ll|'d)?
# |[^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]+[\p{Ll}\p{Lm}\p{Lo}\p{M}]*(?i:'s|'t|'re|'ve|'m|'ll|'d)?
# |\p{N}{1,3}| ?[^\s\p{L}\p{N}]+[\r\n/]*|\s*[\r\n]+|\s+(?!\S)|\s+
O200K = Alt(Seq(opt(NOT_CRLF_L_N), star(UB), plus(LB), opt(CONTRACTION)),
            Seq(opt(NOT_CRLF_L_N), plus(UB), star(LB), opt(CONTRACTION)),
            Rep(NUM, 1, 3),
            Seq(opt(SP), plus(OTHER), star(CRLF_SLASH)),
            Seq(star(WS), plus(CRLF)),
            Seq(plus(WS), NotAhead(NONWS)),
            plus(WS))

PATTERNS = {"gpt2": GPT2, "cl100k": CL100K, "o200k": O200K}


def split(text, pattern):
    node = PATTERNS[pattern]
    out = []
    p = 0
    while p < len(text):
        e = match(node, text, p, lambda q: q)
        assert e is not None and e > p
        out.append((p, e))
        p = e
    return out
