"""The BPE engines on random merge lists, against the oracle.

The stored tables come from one trainer; these merge lists do not.  Random
proper merge lists over a two- and a three-letter alphabet make every unit
one letter run under the GPT-2-style pattern, so units of 1 to 120 bytes
reach the thread, wave and two-row wave engines with merge structures no
trained table has: results of up to 24 or 40 bytes, two results that spell
the same bytes, and a chain a, aa, ..., a^24 under which every substring of
a run of one letter is a token.  Lists over the bytes of multi-byte letters
add byte tokens above 127 and merges inside characters.  Each unit is encoded
as a document of a batch and again inside one request.
"""

import random

import numpy as np
import pytest

from oracle.bpe import MergeTable, bpe

pytestmark = pytest.mark.gpu


def _pack(vocab):
    vb = np.frombuffer(b"".join(vocab), dtype=np.uint8).copy()
    vo = np.zeros(len(vocab) + 1, dtype=np.int64)
    np.cumsum([len(v) for v in vocab], out=vo[1:])
    return vb, vo


def random_merges(seed, letters, n_merges, max_len=24, allow_same_spelling=False):
    """A proper merge list over the bytes of the letters' UTF-8 encodings: each
    merge joins two existing tokens (short ones more often) into a new
    vocabulary entry; a result may hold part of a multi-byte character."""
    rng = random.Random(seed)
    vocab = [bytes([i]) for i in range(256)]
    toks = sorted(set(letters.encode("utf-8")))
    n0 = len(toks)
    spelled = set(vocab)
    pairs = set()
    merges = []
    tries = 0
    while len(merges) < n_merges and tries < 100000:
        tries += 1
        a = rng.choice(toks[: max(n0, len(toks) * rng.choice((1, 2, 4)) // 4)])
        b = rng.choice(toks)
        s = vocab[a] + vocab[b]
        if (a, b) in pairs or len(s) > max_len or (s in spelled and not allow_same_spelling):
            continue
        pairs.add((a, b))
        spelled.add(s)
        vocab.append(s)
        merges.append((a, b, len(vocab) - 1))
        toks.append(len(vocab) - 1)
    return merges, vocab


def _docs(seed, letters, n, lo=1, hi=120):
    rng = random.Random(seed)
    out = []
    for _ in range(n):
        L = rng.randint(lo, hi)
        # runs and repeats, so that long merge results occur in the text
        s = []
        while len(s) < L:
            if s and rng.random() < 0.4:
                k = rng.randint(1, min(len(s), 12))
                s += s[-k:]
            else:
                s.append(rng.choice(letters))
        out.append("".join(s[:L]).encode())
    return out


def _check(merges, vocab, docs):
    from paper_2607_29678_amd import Tokenizer

    table = MergeTable(merges, vocab)
    vb, vo = _pack(vocab)
    with Tokenizer(np.array(merges, dtype=np.int32).reshape(-1, 3), vb, vo, "gpt2") as tok:
        got = tok.encode_batch(docs)
        for d, g in zip(docs, got):
            assert g.tolist() == bpe(d, table), d
        # the same units inside one request, separated by spaces
        req = b" ".join(docs[:400])
        assert tok.encode(req).tolist() == _oracle_request(req, table)


def _oracle_request(req, table):
    from oracle.pretok import pretokenize

    text = req.decode()
    ids = []
    for a, b in pretokenize(text, "gpt2"):
        ids += bpe(text[a:b].encode(), table)
    return ids


@pytest.mark.parametrize("seed,letters,n_merges", [(1, "ab", 300), (2, "ab", 1200), (3, "abc", 800),
                                                    (4, "abc", 3000), (5, "xy", 60)])
def test_random_merge_lists(gpu, seed, letters, n_merges):
    merges, vocab = random_merges(seed, letters, n_merges)
    assert max(len(v) for v in vocab) <= 24
    _check(merges, vocab, _docs(100 + seed, letters, 1500))


@pytest.mark.parametrize("seed,letters,n_merges", [(11, "éж", 600), (12, "aé中", 1500), (13, "ж中😀", 800)])
def test_random_merge_lists_multibyte(gpu, seed, letters, n_merges):
    """Letters of two to four bytes: byte tokens above 127, merges inside and
    across characters, units of up to 240 bytes (the block engine beyond 128),
    and symbol pieces between letter runs where the emoji occurs."""
    merges, vocab = random_merges(seed, letters, n_merges)
    assert any(len(v) > 1 and v[0] >= 0x80 for v in vocab)
    _check(merges, vocab, _docs(300 + seed, letters, 1200, hi=60))


@pytest.mark.parametrize("seed", [6, 7])
def test_results_with_the_same_spelling(gpu, seed):
    """Two merge results spell the same bytes (distinct IDs, distinct pairs)."""
    merges, vocab = random_merges(seed, "ab", 600, allow_same_spelling=True)
    assert len(set(vocab)) < len(vocab)
    _check(merges, vocab, _docs(200 + seed, "ab", 1200))


def test_results_longer_than_the_dictionaries(gpu):
    """Merge results of up to 40 bytes (the whole-unit dictionaries hold 24)."""
    merges, vocab = random_merges(8, "ab", 900, max_len=40)
    assert max(len(v) for v in vocab) > 24
    _check(merges, vocab, _docs(208, "ab", 1200))


def test_runs_of_one_letter_with_every_power_a_token(gpu):
    """Tokens a^2 .. a^24: every substring of a run of the letter a is a token;
    runs of 1..129 letters, and runs followed by another letter."""
    vocab = [bytes([i]) for i in range(256)]
    merges = []
    a = ord("a")
    prev = a
    for k in range(2, 25):
        vocab.append(b"a" * k)
        merges.append((prev, a, len(vocab) - 1))
        prev = len(vocab) - 1
    docs = [b"a" * n for n in range(1, 130)] + [(b"a" * n + b"b") * 3 for n in range(1, 20)]
    _check(merges, vocab, docs)
