"""A small byte-level BPE trainer that makes merge tables from seeded text (oracle; test infrastructure).

The paper encodes with frozen production tables and never trains; the tables
here are synthetic stand-ins with the sizes of the benchmark configurations.
Procedure:

1. pre-tokenize the training text with the same pattern the table will be used
   with, and count the pieces;
2. count adjacent ID pairs inside pieces (overlapping occurrences count), each
   weighted by its piece's count;
3. take the pair with the largest count, ties to the smallest (left, right);
   its result gets the next ID (256 + rank), and every piece applies it to its
   leftmost non-overlapping occurrences;
4. repeat until the requested number of merges, or until no pair is left.
   Pairs with count 1 are taken only when no larger count remains.

Base IDs are the byte values 0..255.  Every operand is a byte or the result of
an earlier merge, so the table is "proper" by construction.

Parity unpinned in the sense of the paper (it is silent on training); the tests
pin determinism, properness and a hand-worked corpus.
"""

import heapq
from collections import Counter

from .pretok import pieces as _pieces


def merge_word(ids, a, b, c):
    """Replace the leftmost non-overlapping occurrences of (a, b) in ``ids`` by ``c``."""
    out = []
    i = 0
    n = len(ids)
    while i < n:
        if i + 1 < n and ids[i] == a and ids[i + 1] == b:
            out.append(c)
            i += 2
        else:
            out.append(ids[i])
            i += 1
    return out


def _pairs(ids):
    return Counter(zip(ids, ids[1:]))


def train_from_counts(piece_counts, n_merges):
    """Merge list [(left, right, result)] learnt from {piece bytes: count}."""
    words = [list(p) for p in piece_counts]
    counts = [piece_counts[p] for p in piece_counts]
    pair_count = Counter()
    where = {}
    for wi, w in enumerate(words):
        c = counts[wi]
        for pr in zip(w, w[1:]):
            pair_count[pr] += c
            where.setdefault(pr, set()).add(wi)
    heap = [(-c, a, b) for (a, b), c in pair_count.items()]
    heapq.heapify(heap)
    merges = []
    while len(merges) < n_merges and heap:
        negc, a, b = heapq.heappop(heap)
        cur = pair_count.get((a, b), 0)
        if cur <= 0 or -negc != cur:
            continue  # stale heap entry
        new = 256 + len(merges)
        merges.append((a, b, new))
        changed = Counter()
        for wi in where.pop((a, b), ()):
            w = words[wi]
            if len(w) < 2:
                continue
            nw = merge_word(w, a, b, new)
            if len(nw) == len(w):
                continue  # index entry was stale
            c = counts[wi]
            old_p = _pairs(w)
            new_p = _pairs(nw)
            for pr, k in old_p.items():
                changed[pr] -= k * c
            for pr, k in new_p.items():
                changed[pr] += k * c
                if pr not in old_p:
                    where.setdefault(pr, set()).add(wi)
            words[wi] = nw
        for pr, d in changed.items():
            if d == 0:
                continue
            v = pair_count[pr] + d
            if v > 0:
                pair_count[pr] = v
                heapq.heappush(heap, (-v, pr[0], pr[1]))
            else:
                pair_count.pop(pr, None)
        pair_count.pop((a, b), None)
    return merges


def vocab_of(merges):
    """ID -> bytes for base bytes 0..255 plus every merge result."""
    vocab = [bytes([i]) for i in range(256)]
    for a, b, c in merges:
        assert c == len(vocab)
        vocab.append(vocab[a] + vocab[b])
    return vocab


def train(text: str, pattern: str, n_merges: int):
    """Merge list and vocabulary learnt from ``text`` pre-tokenized with ``pattern``."""
    counts = Counter(p.encode("utf-8") for p in _pieces(text, pattern))
    merges = train_from_counts(counts, n_merges)
    return merges, vocab_of(merges)
