"""Greedy lowest-rank byte-level BPE for one piece (oracle; test infrastructure).

The model stage encodes each pre-tokenized piece on its own (Appendix,
Definition d:frontend: the model stage is a function of the unit alone;
Lemma l:homo: the encoding of a request is the concatenation of the encodings
of its units).  For byte-level BPE the encoding of a piece is defined by the
merge list: start from the IDs of the piece's single bytes, then repeatedly
replace the adjacent pair with the smallest merge rank by that merge's result,
taking the leftmost occurrence when the same pair occurs more than once, until
no adjacent pair has a rank.

A merge table is an ordered list of ``(left, right, result)`` ID triples; the
list index is the rank (0 = applied first).  The IDs of the 256 single bytes
come from the vocabulary; nothing assumes that ID == byte value.

Two implementations of that one definition, cross-checked by the tests:
``bpe_naive`` scans all pairs on every step; ``bpe_heap`` keeps the candidate
pairs in a heap keyed by (rank, position) over a linked list, for long pieces.
"""

import heapq


class MergeTable:
    """Merge ranks and the single-byte IDs of a vocabulary."""

    def __init__(self, merges, vocab):
        """``merges``: sequence of (left, right, result); ``vocab``: list of bytes, index = ID."""
        self.merges = [tuple(int(x) for x in m) for m in merges]
        self.vocab = [bytes(v) for v in vocab]
        self.rank = {}
        for r, (a, b, c) in enumerate(self.merges):
            if (a, b) in self.rank:
                raise ValueError("duplicate pair (%d, %d)" % (a, b))
            self.rank[(a, b)] = (r, c)
        self.byte_id = [None] * 256
        for i, v in enumerate(self.vocab):
            if len(v) == 1 and self.byte_id[v[0]] is None:
                self.byte_id[v[0]] = i
        if any(x is None for x in self.byte_id):
            raise ValueError("vocabulary lacks a single-byte token")

    def __len__(self):
        return len(self.merges)


def bpe_naive(piece: bytes, table: MergeTable) -> list:
    """IDs of one piece: merge the lowest-ranked adjacent pair, leftmost first, until none is left."""
    ids = [table.byte_id[b] for b in piece]
    rank = table.rank
    while len(ids) > 1:
        best = None
        best_i = -1
        for i in range(len(ids) - 1):
            hit = rank.get((ids[i], ids[i + 1]))
            if hit is not None and (best is None or hit[0] < best[0]):
                best = hit
                best_i = i
        if best is None:
            break
        ids[best_i:best_i + 2] = [best[1]]
    return ids


def bpe_heap(piece: bytes, table: MergeTable, applied=None) -> list:
    """The same definition with a heap of (rank, left position) over a doubly linked list.

    A token keeps the byte position of its first byte, so equal ranks pop in
    left-to-right order, which is the leftmost-first rule.  ``applied``, if
    given, receives the rank of every merge in the order they are applied.
    """
    n = len(piece)
    if n == 0:
        return []
    ids = [table.byte_id[b] for b in piece]
    nxt = list(range(1, n + 1))
    prv = list(range(-1, n - 1))
    alive = [True] * n
    rank = table.rank
    heap = []

    def push(i):
        j = nxt[i]
        if j < n:
            hit = rank.get((ids[i], ids[j]))
            if hit is not None:
                heapq.heappush(heap, (hit[0], i, ids[i], ids[j], hit[1]))

    for i in range(n - 1):
        push(i)
    while heap:
        r, i, a, b, c = heapq.heappop(heap)
        if not alive[i]:
            continue
        j = nxt[i]
        if j >= n or ids[i] != a or ids[j] != b:
            continue  # stale entry: the pair changed after it was pushed
        ids[i] = c
        if applied is not None:
            applied.append(r)
        alive[j] = False
        k = nxt[j]
        nxt[i] = k
        if k < n:
            prv[k] = i
        if prv[i] >= 0:
            push(prv[i])
        push(i)
    out = []
    i = 0
    while i < n:
        out.append(ids[i])
        i = nxt[i]
    return out


NAIVE_MAX = 256


def bpe(piece: bytes, table: MergeTable) -> list:
    """IDs of one piece (naive scan for short pieces, heap above ``NAIVE_MAX`` bytes)."""
    if len(piece) <= NAIVE_MAX:
        return bpe_naive(piece, table)
    return bpe_heap(piece, table)


def bpe_rounds(piece: bytes, table: MergeTable) -> int:
    """Rounds of the round-parallel schedule on one piece (Sec. 4.2: a round
    merges every leftmost non-overlapping occurrence of the lowest-ranked pair
    present).  A merge only creates pairs that hold its result, whose ranks are
    higher in a proper table, so greedy BPE applies its ranks in non-decreasing
    order and each rank in one round: the rounds are the distinct ranks applied.
    The dependency chain of a piece is this many rounds long (Sec. 6: the chain
    depth of exact BPE bounds the GPU's latency)."""
    applied = []
    bpe_heap(piece, table, applied)
    return len(set(applied))
