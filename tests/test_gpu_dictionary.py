"""GPU parity for units that the whole-unit dictionaries resolve.

The library resolves a unit of 3..24 bytes with one lookup when its bytes spell
a token that BPE reproduces from those bytes (a short dictionary up to 12 bytes,
a long one up to 24).  These cases place such spellings as whole pieces in a
text, at every byte alignment, together with near misses (one byte changed),
and as the unit that crosses a tile edge and is encoded by the next tile, and
compare the IDs with the oracle.
"""

import random

import pytest

from conftest import lib_tokenizer, oracle_ids, oracle_table, pattern_of

pytestmark = pytest.mark.gpu

TILE_OWN = 1984  # bytes a tile decides


def _single_token_spellings(k, lo, hi, limit, seed):
    """Valid UTF-8 spellings of lo..hi bytes of merge results whose BPE is that token."""
    from oracle.bpe import bpe

    table = oracle_table(k)
    results = sorted({c for (_r, c) in table.rank.values()})
    cands = [table.vocab[c] for c in results if lo <= len(table.vocab[c]) <= hi]
    rng = random.Random(seed)
    rng.shuffle(cands)
    out = []
    for v in cands:
        try:
            v.decode("utf-8")
        except UnicodeDecodeError:
            continue
        if len(bpe(v, table)) == 1:
            out.append(v)
            if len(out) == limit:
                break
    return out


def _near_miss(v, rng):
    """The spelling with one ASCII letter changed (another letter), if it has one."""
    idx = [i for i, b in enumerate(v) if 97 <= b <= 122]
    if not idx:
        return v + b"q"
    i = rng.choice(idx)
    return v[:i] + bytes([97 + (v[i] - 97 + 1 + rng.randrange(25)) % 26]) + v[i + 1:]


@pytest.mark.parametrize("k", [3, 4])
def test_dictionary_units_parity(gpu, k):
    rng = random.Random(900 + k)
    short = _single_token_spellings(k, 3, 12, 300, 11 * k)
    long_ = _single_token_spellings(k, 13, 24, 300, 13 * k)
    assert len(long_) >= 50, "table %d has few long single-token spellings" % k
    parts = []
    for v in short + long_:
        parts.append(b"\n" * rng.randint(1, 4))  # varies the byte alignment of the unit
        parts.append(v if rng.random() < 0.7 else _near_miss(v, rng))
    data = b"".join(parts) + b"\n"
    got = lib_tokenizer(k).encode(data).tolist()
    want = oracle_ids(data, oracle_table(k), pattern_of(k))
    assert got == want


@pytest.mark.parametrize("k", [3, 4])
def test_dictionary_units_across_tile_edges(gpu, k):
    """A spelling that starts in one tile and ends in the next is the next tile's incoming unit."""
    rng = random.Random(700 + k)
    spell = _single_token_spellings(k, 3, 12, 8, 17 * k) + _single_token_spellings(k, 13, 24, 16, 19 * k)
    filler_words = [b"ab", b"cd", b"ef", b"gh"]
    docs = []
    for v in spell:
        for off in sorted({1, len(v) // 2, len(v) - 1}):
            for edge in (1, 2):
                start = edge * TILE_OWN - off
                body = b" ".join(rng.choice(filler_words) for _ in range(start // 3 + 2))
                filler = body[: start - 1] + b"\n"
                docs.append(filler + v + b"\n" + b"tail words\n")
    tok = lib_tokenizer(k)
    table, pat = oracle_table(k), pattern_of(k)
    memo = {}
    for j, d in enumerate(docs):
        assert tok.encode(d).tolist() == oracle_ids(d, table, pat, memo), "document %d" % j
    got = tok.encode_batch(docs)
    for j, d in enumerate(docs):
        assert got[j].tolist() == oracle_ids(d, table, pat, memo), "batch document %d" % j
