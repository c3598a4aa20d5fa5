"""Write ``workload_shapes.json``: the shape of the benchmark's requests as the
oracle sees them (characters, bytes, pieces, tokens, the longest piece and the
most merge rounds any piece needs), for the first timed 1,000,000-character
sample of C3 and C4 and for the stress request C5 with its 64-document batch.

The benchmark reports these figures next to its timings and checks its token
counts against them.  Run from the repository root:

    python tests/golden/make_workload_shapes.py
"""

import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle.bpe import MergeTable, bpe, bpe_rounds  # noqa: E402
from oracle.pretok import pretokenize  # noqa: E402
from workloads import textgen  # noqa: E402
from workloads.tables import load_table, vocab_list  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "workload_shapes.json")
FIRST_TIMED = 3  # the benchmark warms up on latency samples 0-2


def shape(text, table, pattern):
    memo = {}
    pieces = pretokenize(text, pattern)
    tokens = 0
    longest = 0
    rounds = 0
    for a, b in pieces:
        p = text[a:b].encode("utf-8")
        r = memo.get(p)
        if r is None:
            r = memo[p] = (len(bpe(p, table)), bpe_rounds(p, table))
        tokens += r[0]
        longest = max(longest, len(p))
        rounds = max(rounds, r[1])
    return {"chars": len(text), "bytes": len(text.encode("utf-8")), "pieces": len(pieces), "tokens": tokens,
            "longest_piece_bytes": longest, "max_rounds_per_piece": rounds}


def main():
    out = {}
    for k in (3, 4):
        m, vb, vo = load_table(k)
        t = MergeTable(m.tolist(), vocab_list(vb, vo))
        pat = textgen.CONFIGS[k]["pattern"]
        out["C%d_latency_sample_%d" % (k, FIRST_TIMED)] = shape(textgen.latency_sample(k, FIRST_TIMED), t, pat)
        print(k, out["C%d_latency_sample_%d" % (k, FIRST_TIMED)], flush=True)
    m, vb, vo = load_table(5)
    t = MergeTable(m.tolist(), vocab_list(vb, vo))
    out["C5_request"] = shape(textgen.config_text(5), t, "cl100k")
    print(5, out["C5_request"], flush=True)
    docs = [shape(d, t, "cl100k") for d in textgen.batch_docs()]
    out["C5_batch"] = {"docs": len(docs), "chars": sum(d["chars"] for d in docs), "bytes": sum(d["bytes"] for d in docs),
                       "pieces": sum(d["pieces"] for d in docs), "tokens": sum(d["tokens"] for d in docs),
                       "longest_piece_bytes": max(d["longest_piece_bytes"] for d in docs),
                       "max_rounds_per_piece": max(d["max_rounds_per_piece"] for d in docs)}
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


if __name__ == "__main__":
    main()
