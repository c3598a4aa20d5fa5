"""Pins of the oracle's BPE (CPU only).

  * hand-worked merges, including the case where applying all local minima
    at once would be wrong;
  * the two implementations of the definition (naive scan, heap) agree;
  * the HF tokenizers BPE model with the same merges agrees (library routine);
  * invariants: the IDs spell the input, no adjacent pair inside a piece still
    has a rank, at most one ID per byte;
  * the parallel round schedule the GPU uses (Sec. 4.2: merge every leftmost
    non-overlapping occurrence of the round's lowest-ranked pair) equals the
    greedy definition.
"""

import random

import pytest

from conftest import oracle_table, stored_table
from oracle.bpe import MergeTable, bpe, bpe_heap, bpe_naive, bpe_rounds

# r0 (a,a)->256, r1 (256,a)->257, r2 (a,b)->258, r3 (258,c)->259, r4 (c,d)->260
HAND = [(97, 97, 256), (256, 97, 257), (97, 98, 258), (258, 99, 259), (99, 100, 260)]


def _hand_table():
    vocab = [bytes([i]) for i in range(256)] + [b"aa", b"aaa", b"ab", b"abc", b"cd"]
    return MergeTable(HAND, vocab)


@pytest.mark.parametrize("piece,ids", [
    (b"aaaa", [256, 256]),
    (b"aaaaa", [256, 257]),
    (b"aaab", [257, 98]),
    (b"abcd", [259, 100]),   # all local minima at once would give [258, 260]
    (b"cd", [260]),
    (b"", []),
    (b"x", [120]),
])
def test_hand_worked(piece, ids):
    t = _hand_table()
    assert bpe_naive(piece, t) == ids
    assert bpe_heap(piece, t) == ids


def test_base_ids_not_identity():
    """Relabelled vocabulary: base IDs come from the vocabulary, not from byte values."""
    rng = random.Random(3)
    perm = list(range(261))
    rng.shuffle(perm)
    vocab = [None] * 261
    base = [bytes([i]) for i in range(256)] + [b"aa", b"aaa", b"ab", b"abc", b"cd"]
    for old, new in enumerate(perm):
        vocab[new] = base[old]
    merges = [(perm[a], perm[b], perm[c]) for a, b, c in HAND]
    t = MergeTable(merges, vocab)
    assert bpe(b"abcd", t) == [perm[259], perm[100]]


@pytest.mark.parametrize("k", [1, 2, 3])
def test_naive_equals_heap(k):
    t = oracle_table(k)
    rng = random.Random(k)
    alphabet = b"etaoinshrdlu \n0123456789.,'-_"
    for _ in range(1500):
        p = bytes(rng.choice(alphabet) for _ in range(rng.randint(1, 300)))
        assert bpe_naive(p, t) == bpe_heap(p, t)


def _round_schedule(piece, t):
    ids = [t.byte_id[b] for b in piece]
    while True:
        ranks = [t.rank.get((ids[i], ids[i + 1])) for i in range(len(ids) - 1)]
        present = [r for r in ranks if r is not None]
        if not present:
            return ids
        best = min(present)
        out = []
        i = 0
        while i < len(ids):
            if i + 1 < len(ids) and ranks[i] is not None and ranks[i][0] == best[0]:
                out.append(best[1])
                i += 2
            else:
                out.append(ids[i])
                i += 1
        ids = out


@pytest.mark.parametrize("k", [1, 3])
def test_round_schedule_equals_greedy(k):
    t = oracle_table(k)
    rng = random.Random(10 + k)
    for _ in range(2000):
        p = bytes(rng.choice(b"aaabbcdeet ") for _ in range(rng.randint(1, 60)))
        assert _round_schedule(p, t) == bpe(p, t)


def test_rounds_hand_worked():
    """Rounds of the hand-worked merges: aaaa merges (a, a) twice in one round;
    aaaaa and aaab need (a, a) then (256, a); abcd needs (a, b) then (258, c)."""
    t = _hand_table()
    assert bpe_rounds(b"aaaa", t) == 1
    assert bpe_rounds(b"aaaaa", t) == 2
    assert bpe_rounds(b"aaab", t) == 2
    assert bpe_rounds(b"abcd", t) == 2
    assert bpe_rounds(b"xyz", t) == 0
    assert bpe_rounds(b"", t) == 0


def _rounds_of_schedule(piece, t):
    """Number of rounds the parallel schedule runs (counted by the schedule itself)."""
    ids = [t.byte_id[b] for b in piece]
    rounds = 0
    while True:
        ranks = [t.rank.get((ids[i], ids[i + 1])) for i in range(len(ids) - 1)]
        present = [r for r in ranks if r is not None]
        if not present:
            return rounds
        rounds += 1
        best = min(present)
        out = []
        i = 0
        while i < len(ids):
            if i + 1 < len(ids) and ranks[i] is not None and ranks[i][0] == best[0]:
                out.append(best[1])
                i += 2
            else:
                out.append(ids[i])
                i += 1
        ids = out


@pytest.mark.parametrize("k", [1, 3])
def test_rounds_equal_the_schedule(k):
    """The distinct ranks greedy BPE applies equal the rounds of the parallel schedule."""
    t = oracle_table(k)
    rng = random.Random(20 + k)
    for _ in range(1500):
        p = bytes(rng.choice(b"aaabbcdeet ") for _ in range(rng.randint(1, 80)))
        assert bpe_rounds(p, t) == _rounds_of_schedule(p, t)


def test_planted_fault_is_caught():
    """Harness validation: plausible wrong variants of the definition fail the hand-worked pins."""
    t = _hand_table()

    def rightmost_first(piece):
        ids = [t.byte_id[b] for b in piece]
        while True:
            best = None
            for i in range(len(ids) - 1):
                h = t.rank.get((ids[i], ids[i + 1]))
                if h is not None and (best is None or h[0] <= best[0][0]):
                    best = (h, i)
            if best is None:
                return ids
            ids[best[1]:best[1] + 2] = [best[0][1]]

    def all_local_minima(piece):
        return _round_schedule_local(piece, t)

    assert rightmost_first(b"aaab") != [257, 98]
    assert all_local_minima(b"abcd") != [259, 100]


def _round_schedule_local(piece, t):
    """Wrong on purpose: merges every pair whose rank is below both neighbours' in one step."""
    ids = [t.byte_id[b] for b in piece]
    while True:
        r = [t.rank.get((ids[i], ids[i + 1]), (1 << 40, None))[0] for i in range(len(ids) - 1)]
        pick = [i for i in range(len(r)) if r[i] < (1 << 40) and (i == 0 or r[i] < r[i - 1])
                and (i + 1 == len(r) or r[i] < r[i + 1])]
        if not pick:
            return ids
        out = []
        i = 0
        while i < len(ids):
            if i in pick:
                out.append(t.rank[(ids[i], ids[i + 1])][1])
                i += 2
            else:
                out.append(ids[i])
                i += 1
        ids = out


@pytest.mark.parametrize("k", [1, 2])
def test_invariants_on_text(k):
    from conftest import config_bytes, pattern_of
    from oracle.pretok import pretokenize

    t = oracle_table(k)
    text = config_bytes(k).decode("utf-8")
    for a, b in pretokenize(text, pattern_of(k))[:20000]:
        p = text[a:b].encode("utf-8")
        ids = bpe(p, t)
        assert b"".join(t.vocab[i] for i in ids) == p
        assert len(ids) <= len(p)
        assert all((ids[i], ids[i + 1]) not in t.rank for i in range(len(ids) - 1))


def _bytes_to_unicode():
    bs = list(range(ord("!"), ord("~") + 1)) + list(range(ord("¡"), ord("¬") + 1)) + list(range(ord("®"), ord("ÿ") + 1))
    cs = bs[:]
    n = 0
    for b in range(256):
        if b not in bs:
            bs.append(b)
            cs.append(256 + n)
            n += 1
    return {b: chr(c) for b, c in zip(bs, cs)}


@pytest.mark.parametrize("k", [1, 2])
def test_against_hf_bpe(k):
    tk = pytest.importorskip("tokenizers")
    m, _, _ = stored_table(k)
    t = oracle_table(k)
    b2u = _bytes_to_unicode()

    def s(tok):
        return "".join(b2u[x] for x in t.vocab[tok])

    strings = [s(i) for i in range(len(t.vocab))]
    if len(set(strings)) != len(strings):
        pytest.skip("table has duplicate byte strings; the HF model cannot represent it")
    vocab = {st: i for i, st in enumerate(strings)}
    merges = [(s(a), s(b)) for a, b, _ in m.tolist()]
    model = tk.models.BPE(vocab=vocab, merges=merges)
    rng = random.Random(k)
    alphabet = b"etaoinshrdlu \n0123456789"
    for _ in range(2000):
        p = bytes(rng.choice(alphabet) for _ in range(rng.randint(1, 40)))
        hf = [tok.id for tok in model.tokenize("".join(b2u[x] for x in p))]
        assert hf == bpe(p, t), p


def _junctions(t):
    return {(t.vocab[a][-1], t.vocab[b][0]) for a, b, _ in t.merges}


def _segments(piece, junctions):
    out, prev = [], 0
    for i in range(1, len(piece)):
        if (piece[i - 1], piece[i]) not in junctions:
            out.append(piece[prev:i])
            prev = i
    out.append(piece[prev:])
    return out


@pytest.mark.parametrize("k", [1, 3, 4])
def test_junction_barrier_segments_encode_independently(k):
    """A byte boundary whose byte pair is the junction of no merge is never crossed by any merge,
    so BPE of the piece equals BPE of the segments between such boundaries, concatenated (the
    library cuts pieces there before BPE)."""
    from conftest import config_bytes, pattern_of
    from oracle.pretok import pretokenize

    t = oracle_table(k)
    jn = _junctions(t)
    text = config_bytes(k).decode("utf-8")
    spans = pretokenize(text, pattern_of(k))
    rng = random.Random(k)
    for a, b in rng.sample(spans, min(5000, len(spans))):
        p = text[a:b].encode("utf-8")
        assert sum((bpe(s, t) for s in _segments(p, jn)), []) == bpe(p, t)


def test_junction_barriers_on_random_tables():
    rng = random.Random(5)
    for trial in range(30):
        alphabet = b"abcd"
        vocab = [bytes([i]) for i in range(256)]
        merges = []
        for r in range(rng.randint(1, 12)):
            a = rng.choice(list(alphabet) + list(range(256, len(vocab))))
            b = rng.choice(list(alphabet) + list(range(256, len(vocab))))
            if any(m[0] == a and m[1] == b for m in merges):
                continue
            merges.append((a, b, len(vocab)))
            vocab.append(vocab[a] + vocab[b])
        t = MergeTable(merges, vocab)
        jn = _junctions(t)
        for _ in range(300):
            p = bytes(rng.choice(alphabet) for _ in range(rng.randint(1, 30)))
            assert sum((bpe(s, t) for s in _segments(p, jn)), []) == bpe(p, t), (merges, p)
