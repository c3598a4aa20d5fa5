"""Write ``onig_o200k_classes.txt``: the letter and mark sub-classes the o200k-style pattern sees.

The o200k-style pattern tells upper-case letters from lower-case ones and
treats combining marks as letter material (Sec. 4.1: the o200k lineage adds
a case-boundary rule, and Unicode marks need care).  Its character sets are
built from the general categories Lu, Lt, Ll, Lm, Lo and M.  As for the other
classes, these are probed out of the reference engine (Oniguruma in HF
``tokenizers`` 0.22.2) rather than taken from a library's Unicode data.

Classes written (every other scalar value keeps its class from
``onig_classes.txt``):
  UP  \\p{Lu} or \\p{Lt}     (only in the upper-case letter set)
  LO  \\p{Ll}               (only in the lower-case letter set)
  BO  \\p{Lm} or \\p{Lo}     (in both letter sets)
  MK  \\p{M}                (in both letter sets, and in the "not letter, not
                            number" sets)

Run:  python oracle/data/probe_onig_o200k.py   (needs ``tokenizers``; a few seconds)
"""

import os

from tokenizers import __version__

from probe_onig import matched, scalar_values

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "onig_o200k_classes.txt")


def probe():
    cps = scalar_values()
    text = "".join(chr(c) for c in cps)
    cls = {}
    for name, pats in (("UP", [r"\p{Lu}", r"\p{Lt}"]), ("LO", [r"\p{Ll}"]), ("BO", [r"\p{Lm}", r"\p{Lo}"]),
                       ("MK", [r"\p{M}"])):
        for pat in pats:
            for c in matched(pat, cps, text):
                assert cls.get(c, name) == name, "sub-classes overlap at U+%04X" % c
                cls[c] = name
    letters = set(matched(r"\p{L}", cps, text))
    assert letters == {c for c, k in cls.items() if k != "MK"}, "Lu/Lt/Ll/Lm/Lo do not make up \\p{L}"
    return cls


def main():
    cls = probe()
    lines = [
        "# Letter and mark sub-classes of the o200k-style pattern, probed from Oniguruma in",
        "# HF tokenizers %s.  UP = Lu|Lt, LO = Ll, BO = Lm|Lo, MK = M." % __version__,
        "# Range lines: <first> <last> <class>, hex, inclusive.",
    ]
    run = None
    for c in range(0x110001):
        k = cls.get(c) if c < 0x110000 else None
        if run and (k != run[2] or c != run[1] + 1):
            lines.append("%04X %04X %s" % run)
            run = None
        if k is not None:
            run = (run[0], c, k) if run else (c, c, k)
    with open(OUT, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("wrote %s: %d code points" % (OUT, len(cls)))


if __name__ == "__main__":
    main()
