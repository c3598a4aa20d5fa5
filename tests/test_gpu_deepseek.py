"""The DeepSeek-style pattern (three splitters in sequence) on the GPU, against the oracle.

The pattern has no stored table of its own: the multilingual table (100,000
merges) serves it, since ID parity does not depend on how a table was trained.
Split level and ID level are compared on the seeded texts, on fuzz strings
over an alphabet with every class the splitters distinguish (ASCII and other
letters, marks, numbers, ASCII and other punctuation and symbols, U+0020,
other whitespace, CR/LF, control characters, and letters, marks, symbols and
unassigned code points of the CJK/kana ranges), and on long runs placed across
tile edges, which exercise the walks that start in the previous tile and the
grouping of numbers in threes from the head of their run.
"""

import random

import numpy as np
import pytest

from conftest import config_bytes, oracle_ids, oracle_table, stored_table
from oracle.added import encode_ex
from oracle.pretok import piece_byte_starts

pytestmark = pytest.mark.gpu

_TOK = {}


def _tok(ignore=False, added=None):
    from paper_2607_29678_amd import Tokenizer

    key = (ignore, tuple(added or ()))
    if key not in _TOK:
        m, vb, vo = stored_table(4)
        _TOK[key] = Tokenizer(m, vb, vo, "deepseek", ignore_merges=ignore, added=added)
    return _TOK[key]


def _first_diff(a, b):
    for i in range(min(len(a), len(b))):
        if a[i] != b[i]:
            return i
    return -1 if len(a) == len(b) else min(len(a), len(b))


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_split_parity_seeded(gpu, k):
    data = config_bytes(k)
    got = _tok().pretokenize(data).tolist()
    want = piece_byte_starts(data.decode(), "deepseek")
    d = _first_diff(got, want)
    assert d == -1, "C%d: first piece difference at %d: %s vs %s" % (k, d, got[d:d + 3], want[d:d + 3])


@pytest.mark.parametrize("k", [3, 4])
def test_id_parity_seeded(gpu, k):
    data = config_bytes(k)
    got = _tok().encode(data).tolist()
    want = oracle_ids(data, oracle_table(4), "deepseek")
    d = _first_diff(got, want)
    assert d == -1, "C%d: first ID difference at %d of %d/%d" % (k, d, len(got), len(want))


ALPHA = (list("aAbBsStTdD1 \n\r\t'./-_") + ["中", "文", "ʰ", "́", "̈", "ǅ", "É",
                                             "ä", "ſ", "А", "а", "。", " ", "\u0085",
                                             "²", "\U0001f600"])


def _fuzz(seed, n, max_len):
    rng = random.Random(seed)
    return ["".join(rng.choice(ALPHA) for _ in range(rng.randint(0, max_len))) for _ in range(n)]


def test_fuzz_batch_parity(gpu):
    docs = _fuzz(0x0200, 4000, 24)
    got = _tok().encode_batch([d.encode() for d in docs])
    memo = {}
    table = oracle_table(4)
    for d, g in zip(docs, got):
        assert g.tolist() == oracle_ids(d.encode(), table, "deepseek", memo), repr(d)


def test_fuzz_split_parity(gpu):
    tok = _tok()
    for s in _fuzz(0x0201, 400, 48):
        d = s.encode()
        assert tok.pretokenize(d).tolist() == piece_byte_starts(s, "deepseek"), repr(s)


def _runs(rng):
    """Long runs that keep a segment open across tile edges."""
    letters = "".join(rng.choice("abcdefghij") for _ in range(3000))
    caps = "".join(rng.choice("ABCDEFGH") for _ in range(3000))
    cjk_caps = "".join(rng.choice(["中", "A", "B", "文"]) for _ in range(1500))
    marks = "".join(rng.choice(["a", "́", "B", "̈"]) for _ in range(2000))
    syms = "".join(rng.choice(["/", ".", "\n", "-", "\r"]) for _ in range(2500))
    spaces = "".join(rng.choice([" ", "\t", "\n", " "]) for _ in range(2500))
    digits = "".join(rng.choice("0123456789") for _ in range(2500))
    return [letters, caps, cjk_caps, marks, syms, spaces, digits, caps + "x", cjk_caps + ".", marks + "'S"]


def test_long_runs_across_tile_edges(gpu):
    """Runs of 1,500-3,000 characters starting at several offsets before a tile
    edge (tiles own 1,984 bytes), followed by ordinary text."""
    rng = random.Random(9)
    tok = _tok()
    table = oracle_table(4)
    docs = []
    for run in _runs(rng):
        for off in (1, 31, 32, 33, 500, 1983):
            pre = ("Ab. " * 600)[:1984 - off]
            docs.append((pre + run + " tail Word").encode())
    for d in docs:
        s = d.decode()
        assert tok.pretokenize(d).tolist() == piece_byte_starts(s, "deepseek"), s[1900:2100]
        assert tok.encode(d).tolist() == oracle_ids(d, table, "deepseek")
    got = tok.encode_batch(docs)
    for d, g in zip(docs, got):
        assert g.tolist() == oracle_ids(d, table, "deepseek")


def test_spans_sessions_and_options(gpu):
    from oracle.spans import spans_of
    from paper_2607_29678_amd import Session

    table = oracle_table(4)
    text = config_bytes(4).decode()[:40000]
    data = text.encode()
    ids, spans = _tok().encode_spans(data)
    want = oracle_ids(data, table, "deepseek")
    assert ids.tolist() == want
    assert [tuple(x) for x in spans.tolist()] == [tuple(x) for x in spans_of(want, data, table)]
    # a session appended in random chunks
    sess = Session(_tok())
    rng = random.Random(4)
    pos = 0
    while pos < len(text):
        nxt = min(len(text), pos + rng.randint(1, 1200))
        sess.append(text[pos:nxt].encode())
        pos = nxt
        assert sess.ids().tolist() == oracle_ids(text[:pos].encode(), table, "deepseek")
    sess.close()
    # ignore_merges and literals
    lits = [("<｜end▁of▁sentence｜>", 200000), ("<|im_start|>", 200001)]
    s = text[:5000] + "<|im_start|>" + text[5000:9000] + "<｜end▁of▁sentence｜>"
    for ignore in (False, True):
        got = _tok(ignore, lits).encode(s.encode()).tolist()
        assert got == encode_ex(s.encode(), table, "deepseek", [(a.encode(), i) for a, i in lits], ignore)
