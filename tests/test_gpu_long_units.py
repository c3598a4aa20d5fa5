"""GPU parity for long BPE units and tile-boundary placements.

The library encodes a unit (a piece, or a part of a piece that no merge can
join across) with one thread up to 16 bytes, half a wave up to 32 bytes (two
such units share a wave), one wave up to 64 bytes, the whole block over rows in
LDS up to a tile window, and over rows in global memory beyond that; a unit that starts in one tile and ends in a later one is
encoded by the later tile.  These cases build units of chosen lengths from
bytes whose every adjacent pair is the junction of some merge (so nothing cuts
them), put them at chosen offsets from the tile edges, and compare the IDs with
the oracle.
"""

import random

import pytest

from conftest import lib_tokenizer, oracle_ids, oracle_table, pattern_of

pytestmark = pytest.mark.gpu

TILE_OWN = 1984  # bytes a tile decides (a 2,048-byte window less 32 bytes of context each side)


def _junctions(k):
    table = oracle_table(k)
    out = set()
    for (a, b) in table.rank:
        va, vb = table.vocab[a], table.vocab[b]
        out.add((va[-1], vb[0]))
    return out


def _clique(k, candidates):
    """Bytes from `candidates` whose every ordered pair (including x, x) is a junction."""
    j = _junctions(k)
    chosen = []
    for c in candidates:
        if (c, c) in j and all((c, d) in j and (d, c) in j for d in chosen):
            chosen.append(c)
    return chosen


def _long_texts(k, seed):
    rng = random.Random(seed)
    letters = _clique(k, b"etaoinsrhldcumfpgwybvkxjqz")
    spaces = _clique(k, b" ")
    assert len(letters) >= 2, "table %d has no two-letter junction clique" % k
    texts = []
    for n in (17, 40, 63, 64, 65, 100, 127, 128, 129, 300, 479, 480, 481, 700, 1000, 1500, 2000, 2047, 2048, 2049,
              2100, 3000, 5000):
        body = bytes(rng.choice(letters) for _ in range(n))
        texts.append(b"x " + body + b" y")
        texts.append(body)
    if spaces:
        for n in (20, 70, 500, 2500):
            texts.append(b"a" + b" " * n + b"b")
    # long units placed across tile edges
    for edge in (1, 2, 3):
        for off in (-70, -40, -5, -1, 0, 1, 5, 33):
            pre = edge * TILE_OWN + off
            filler = " ".join("ab" for _ in range(max(0, pre) // 3 + 1)).encode()[: max(0, pre)]
            body = bytes(rng.choice(letters) for _ in range(rng.choice((30, 90, 400, 2300))))
            texts.append(filler + body + b". end")
    return texts


@pytest.mark.parametrize("k", [1, 4])
def test_long_units_id_parity(gpu, k):
    tok = lib_tokenizer(k)
    memo = {}
    for i, data in enumerate(_long_texts(k, 77 + k)):
        got = tok.encode(data).tolist()
        want = oracle_ids(data, oracle_table(k), pattern_of(k), memo)
        assert got == want, "case %d: %d bytes" % (i, len(data))


@pytest.mark.parametrize("k", [1, 4])
def test_long_units_batch_parity(gpu, k):
    docs = _long_texts(k, 177 + k)
    got = lib_tokenizer(k).encode_batch(docs)
    memo = {}
    for j, d in enumerate(docs):
        assert got[j].tolist() == oracle_ids(d, oracle_table(k), pattern_of(k), memo), "document %d" % j


@pytest.mark.parametrize("k", [2, 4])
def test_lengths_around_tile_edges(gpu, k):
    """Prefixes of a seeded config text cut at lengths around multiples of the tile size."""
    from conftest import config_bytes

    text = config_bytes(k)
    tok = lib_tokenizer(k)
    memo = {}
    for edge in (1, 2, 5):
        for off in (-3, -1, 0, 1, 2, 31, 32, 33):
            n = edge * TILE_OWN + off
            while n > 0 and (text[n] & 0xC0) == 0x80:  # cut at a character boundary
                n -= 1
            data = text[:n]
            got = tok.encode(data).tolist()
            want = oracle_ids(data, oracle_table(k), pattern_of(k), memo)
            assert got == want, "length %d" % n


def _paired_texts(k, seed):
    """Many units of 17-32 bytes (two share a wave, one per half), mixed with
    longer ones that go first in the queue, odd and even counts per tile, and
    such units at tile edges, where one of a pair is the tile's incoming unit."""
    rng = random.Random(seed)
    letters = _clique(k, b"etaoinsrhldcumfpgwybvkxjqz")
    texts = []

    def unit(n):
        return bytes(rng.choice(letters) for _ in range(n))

    for count in (1, 2, 3, 7, 8, 9, 40, 41, 150):
        parts = [unit(rng.choice((17, 18, 24, 25, 31, 32))) for _ in range(count)]
        parts += [unit(rng.choice((33, 48, 64, 65, 100))) for _ in range(count // 3)]
        rng.shuffle(parts)
        texts.append(b" ".join(parts))
    for edge in (1, 2):
        for off in (-20, -17, -1, 0, 3):
            pre = edge * TILE_OWN + off
            filler = b" ".join(unit(rng.choice((17, 20, 32))) for _ in range(max(1, pre // 22)))[: max(0, pre)]
            texts.append(filler + unit(rng.choice((17, 23, 32))) + b" " + unit(19) + b" z")
    return texts


@pytest.mark.parametrize("k", [1, 4])
def test_paired_wave_units(gpu, k):
    tok = lib_tokenizer(k)
    memo = {}
    texts = _paired_texts(k, 91 + k)
    for i, data in enumerate(texts):
        got = tok.encode(data).tolist()
        want = oracle_ids(data, oracle_table(k), pattern_of(k), memo)
        assert got == want, "case %d: %d bytes" % (i, len(data))
    got = tok.encode_batch(texts)
    for j, d in enumerate(texts):
        assert got[j].tolist() == oracle_ids(d, oracle_table(k), pattern_of(k), memo), "document %d" % j
