"""Train the merge tables of the benchmark configurations and store them (oracle; test infrastructure).

Writes ``workloads/tables/c<k>.npz`` for k = 1..4 (configuration 5 uses the
table of configuration 4).  Each file holds

* ``merges``         int32 [M, 3]  (left, right, result); row index = rank
* ``vocab_bytes``    uint8 [sum of token lengths]  token byte strings, concatenated
* ``vocab_offsets``  int64 [V + 1]  token i spans vocab_bytes[off[i]:off[i+1]]

Only this script writes those files, and it calls nothing but ``oracle`` and
the seeded text generator.

Run:  python -m oracle.train_tables [k ...]      (k = 3 and 4 take a few minutes each)
"""

import hashlib
import os
import sys
import time

import numpy as np

from workloads import textgen
from workloads.tables import TABLE_DIR

from .train import train


def pack(merges, vocab):
    m = np.asarray(merges, dtype=np.int32).reshape(-1, 3)
    lens = np.array([len(v) for v in vocab], dtype=np.int64)
    off = np.zeros(len(vocab) + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    vb = np.frombuffer(b"".join(vocab), dtype=np.uint8)
    return m, vb, off


def main(argv):
    ks = [int(a) for a in argv] or [1, 2, 3, 4]
    os.makedirs(TABLE_DIR, exist_ok=True)
    for k in ks:
        cfg = textgen.CONFIGS[k]
        t0 = time.time()
        text = textgen.training_text(k)
        merges, vocab = train(text, cfg["pattern"], cfg["merges"])
        m, vb, off = pack(merges, vocab)
        path = os.path.join(TABLE_DIR, "c%d.npz" % k)
        np.savez_compressed(path, merges=m, vocab_bytes=vb, vocab_offsets=off)
        digest = hashlib.sha256(m.tobytes()).hexdigest()
        print("c%d: %d merges (asked %d), %.1fs, merges sha256 %s" % (
            k, len(merges), cfg["merges"], time.time() - t0, digest), file=sys.stderr)


if __name__ == "__main__":
    main(sys.argv[1:])
