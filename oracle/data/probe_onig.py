"""Write ``onig_classes.txt``: the character classes the patterns see, probed from the regex engine.

The paper pins its Unicode class tables by probing them out of the reference
engine instead of taking them from a library's Unicode data, because two
Unicode versions disagreed on thousands of code points (Sec. 4.1 on table
pinning; Sec. 5.2 on the table skew it found).  The reference engine here is
the Oniguruma build inside HF ``tokenizers`` 0.22.2, the version the paper
pins.  This script asks that engine, for every Unicode scalar value, whether it
matches ``\\p{L}``, ``\\p{N}`` and ``\\s``, and which code points match each
contraction letter case-insensitively.

Run:  python oracle/data/probe_onig.py   (needs ``tokenizers``; a few seconds)
"""

import os
import sys

from tokenizers import Regex, __version__, pre_tokenizers

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "onig_classes.txt")


def scalar_values():
    return [c for c in range(0x110000) if not 0xD800 <= c <= 0xDFFF]


def matched(pattern, cps, text):
    """Code points of ``cps`` (one per char of ``text``) that ``pattern`` matches."""
    split = pre_tokenizers.Split(Regex(pattern), behavior="removed")
    left = set()
    for _, (a, b) in split.pre_tokenize_str(text):
        left.update(range(a, b))
    return [cps[i] for i in range(len(cps)) if i not in left]


def probe():
    cps = scalar_values()
    text = "".join(chr(c) for c in cps)
    cls = {}
    for name, pat in (("L", r"\p{L}"), ("N", r"\p{N}"), ("W", r"\s")):
        for c in matched(pat, cps, text):
            assert c not in cls, "classes overlap at U+%04X" % c
            cls[c] = name
    folds = {}
    for letter in "strevmld":
        folds[letter] = matched("(?i:%s)" % letter, cps, text)
    return cls, folds


def main():
    cls, folds = probe()
    lines = [
        "# Character classes of the pre-tokenization patterns, probed from Oniguruma in",
        "# HF tokenizers %s.  L = \\p{L}, N = \\p{N}, W = \\s; every other scalar value is O." % __version__,
        "# Range lines: <first> <last> <class>, hex, inclusive.",
        "# FOLD lines: <letter> <code points matching it case-insensitively>.",
    ]
    run = None
    for c in range(0x110000):
        k = cls.get(c)
        if run and run[2] == k and run[1] == c - 1:
            run[1] = c
            continue
        if run and run[2] is not None:
            lines.append("%04X %04X %s" % tuple(run))
        run = [c, c, k]
    if run and run[2] is not None:
        lines.append("%04X %04X %s" % tuple(run))
    for letter in "strevmld":
        lines.append("FOLD %s %s" % (letter, " ".join("%04X" % c for c in folds[letter])))
    with open(OUT, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("wrote", OUT, len(lines), "lines", file=sys.stderr)


if __name__ == "__main__":
    main()
