"""Write ``onig_deepseek_classes.txt``: the punctuation and symbol code points.

The DeepSeek-style pattern's third splitter tests the general categories P
(punctuation) and S (symbols) besides letters, marks, numbers and whitespace
(Sec. 4.1: DeepSeek-family tokenizers apply three splitters in sequence).  As
for the other classes, these are probed out of the reference engine
(Oniguruma in HF ``tokenizers`` 0.22.2) rather than taken from a library's
Unicode data.

Class written (every other scalar value keeps its classes from
``onig_classes.txt`` and ``onig_o200k_classes.txt``):
  PS  \\p{P} or \\p{S}

Run:  python oracle/data/probe_onig_deepseek.py   (needs ``tokenizers``; a few seconds)
"""

import os

from tokenizers import __version__

from probe_onig import matched, scalar_values

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "onig_deepseek_classes.txt")


def probe():
    cps = scalar_values()
    text = "".join(chr(c) for c in cps)
    ps = set(matched(r"\p{P}", cps, text)) | set(matched(r"\p{S}", cps, text))
    both = set(matched(r"[\p{P}\p{S}]", cps, text))
    assert ps == both, "the class union disagrees with the two categories"
    return sorted(ps)


def main():
    ps = probe()
    lines = [
        "# Punctuation and symbol code points of the DeepSeek-style pattern, probed from",
        "# Oniguruma in HF tokenizers %s.  PS = \\p{P} or \\p{S}." % __version__,
        "# Range lines: <first> <last> <class>, hex, inclusive.",
    ]
    run = None
    for c in ps + [None]:
        if run and (c is None or c != run[1] + 1):
            lines.append("%04X %04X PS" % tuple(run))
            run = None
        if c is not None:
            run = [run[0], c] if run else [c, c]
    with open(OUT, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("wrote %s: %d code points" % (OUT, len(ps)))


if __name__ == "__main__":
    main()
