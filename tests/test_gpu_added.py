"""ignore_merges and added-token literals on the GPU, against the oracle.

The oracle (``oracle.added.encode_ex``) is pinned to HF tokenizers in
``test_oracle_added.py``.  The stored tables are self-consistent (every entry's
BPE is the entry itself), so on them ignore_merges only exercises the probe
path; the tables below add vocabulary entries that no merge produces (short,
long and longer than the probe tables' embedded keys) and a merge order under
which an entry's BPE is not the entry, so that the probe changes the result.
"""

import random

import numpy as np
import pytest

from conftest import config_bytes, oracle_table, pattern_of, stored_table
from oracle.added import encode_ex
from oracle.bpe import MergeTable, bpe
from oracle.pretok import pretokenize
from oracle.spans import spans_of

pytestmark = pytest.mark.gpu


def _pack(vocab):
    vb = np.frombuffer(b"".join(vocab), dtype=np.uint8).copy()
    vo = np.zeros(len(vocab) + 1, dtype=np.int64)
    np.cumsum([len(v) for v in vocab], out=vo[1:])
    return vb, vo


_EXT = {}


def extended_table(k):
    """Table k plus extra vocabulary entries: spellings of pieces of the config
    text that BPE splits into several tokens (2..60 bytes, so that the probe
    tables of every length class are used) and a few long whitespace and
    punctuation runs.  Merges are unchanged."""
    if k in _EXT:
        return _EXT[k]
    m, _, _ = stored_table(k)
    t = oracle_table(k)
    vocab = list(t.vocab)
    have = set(vocab)
    text = config_bytes(k).decode()
    extra = []
    for a, b in pretokenize(text, pattern_of(k)):
        p = text[a:b].encode()
        if 2 <= len(p) <= 60 and p not in have and len(bpe(p, t)) >= 2:
            have.add(p)
            extra.append(p)
    for p in [b" " * 40, b"\n" * 30, b"-" * 33, b"=" * 64, b" " * 7]:
        if p not in have:
            have.add(p)
            extra.append(p)
    vocab += extra
    table = MergeTable(m.tolist(), vocab)
    vb, vo = _pack(vocab)
    _EXT[k] = (m, vb, vo, table, extra)
    return _EXT[k]


def _tok(m, vb, vo, pattern, ignore, added=None):
    from paper_2607_29678_amd import Tokenizer

    return Tokenizer(m, vb, vo, pattern, ignore_merges=ignore, added=added)


@pytest.mark.parametrize("k", [1, 2, 4])
def test_ignore_merges_stored_tables(gpu, k):
    m, vb, vo = stored_table(k)
    data = config_bytes(k)
    with _tok(m, vb, vo, pattern_of(k), True) as tok:
        got = tok.encode(data).tolist()
    assert got == encode_ex(data, oracle_table(k), pattern_of(k), ignore_merges=True)


@pytest.mark.parametrize("k", [1, 4])
def test_ignore_merges_extra_entries(gpu, k):
    """Entries no merge produces become the pieces' IDs; without the option the
    same handle tables give plain BPE."""
    m, vb, vo, table, extra = extended_table(k)
    assert len(extra) > 50
    pat = pattern_of(k)
    data = config_bytes(k)
    want = encode_ex(data, table, pat, ignore_merges=True)
    assert want != encode_ex(data, table, pat, ignore_merges=False)
    with _tok(m, vb, vo, pat, True) as tok:
        assert tok.encode(data).tolist() == want
        # every extra entry alone, after a space and inside text
        docs = []
        for e in extra[:300]:
            s = e.decode()
            docs += [e, (" " + s).encode(), ("x." + s + " y").encode()]
        got = tok.encode_batch(docs)
        for d, g in zip(docs, got):
            assert g.tolist() == encode_ex(d, table, pat, ignore_merges=True), d
    with _tok(m, vb, vo, pat, False) as tok:
        assert tok.encode(data).tolist() == encode_ex(data, table, pat, ignore_merges=False)


def test_ignore_merges_pieces_across_tile_edges(gpu):
    """Whole-vocabulary pieces of 2..64 bytes placed across every offset of a
    tile edge (tiles own 1,984 bytes): the tile's last piece goes to the next
    tile whole and is probed there."""
    m, vb, vo, table, extra = extended_table(1)
    longs = sorted(extra, key=len)[-40:] + [b"=" * 64, b"-" * 33]
    rng = random.Random(5)
    docs = []
    for e in longs:
        for off in (1, 2, 7, 30, 31, 32, 33, len(e) - 1):
            pre = 1984 - off
            filler = ("ab. " * 600)[:pre]
            docs.append(filler.encode() + e + b" tail")
    rng.shuffle(docs)
    with _tok(m, vb, vo, "gpt2", True) as tok:
        for d in docs:
            assert tok.encode(d).tolist() == encode_ex(d, table, "gpt2", ignore_merges=True), d[1900:2100]
        got = tok.encode_batch(docs)
    for d, g in zip(docs, got):
        assert g.tolist() == encode_ex(d, table, "gpt2", ignore_merges=True)


def test_ignore_merges_changes_bpe_order(gpu):
    """A merge list under which the entry "abc" is not its own BPE."""
    vocab = [bytes([i]) for i in range(256)] + [b"bc", b"ab", b"abc"]
    a, b, c = ord("a"), ord("b"), ord("c")
    merges = [(b, c, 256), (a, b, 257), (257, c, 258)]
    table = MergeTable(merges, vocab)
    vb, vo = _pack(vocab)
    texts = [b"abc", b"abc abc", b"xabc", b"abcabc", b"ab c abc\nabc", b"'abc", b"abcd"]
    for pat in ("gpt2", "cl100k"):
        with _tok(merges, vb, vo, pat, True) as tok:
            for s in texts:
                assert tok.encode(s).tolist() == encode_ex(s, table, pat, ignore_merges=True), s
        with _tok(merges, vb, vo, pat, False) as tok:
            assert tok.encode(b"abc").tolist() == [a, 256]


@pytest.mark.parametrize("k", [1, 4])
def test_ignore_merges_spans_and_sessions(gpu, k):
    from paper_2607_29678_amd import Session

    m, vb, vo, table, extra = extended_table(k)
    pat = pattern_of(k)
    data = config_bytes(k)[:30000]
    text = data.decode()
    want = encode_ex(data, table, pat, ignore_merges=True)
    with _tok(m, vb, vo, pat, True) as tok:
        ids, spans = tok.encode_spans(data)
        assert ids.tolist() == want
        assert [tuple(x) for x in spans.tolist()] == [tuple(x) for x in spans_of(want, data, table)]
        sess = Session(tok)
        rng = random.Random(k)
        pos = 0
        while pos < len(text):
            nxt = min(len(text), pos + rng.randint(1, 900))
            sess.append(text[pos:nxt].encode())
            pos = nxt
            assert sess.ids().tolist() == encode_ex(text[:pos].encode(), table, pat, ignore_merges=True)
        sess.close()


LITERALS = ["<|endoftext|>", "<|im_start|>", "<|im_end|>", "<|e", "<|end", "[INST]", "é<é>", "\n\n<sep>",
            "<|reserved_special_token_123|>"]


def _with_literals(text, rng, n):
    parts = []
    a = rng.randint(0, len(text) // 2)
    for _ in range(n):
        parts.append(text[a:a + rng.randint(0, 80)])
        a += 80
        parts.append(rng.choice(LITERALS + ["<|", "|>", "<|im_", "é<", "<é>"]))
    parts.append(text[a:a + rng.randint(0, 80)])
    return "".join(parts)


@pytest.mark.parametrize("k,ignore", [(1, False), (4, False), (4, True)])
def test_added_tokens(gpu, k, ignore):
    pat = pattern_of(k)
    m, vb, vo = stored_table(k)
    table = oracle_table(k)
    lits = [(x, 300000 + i) for i, x in enumerate(LITERALS)]
    olits = [(x.encode(), i) for x, i in lits]
    text = config_bytes(k).decode()
    rng = random.Random(11 * k + ignore)
    with _tok(m, vb, vo, pat, ignore, lits) as tok:
        # single requests: short and long, literals at the edges and adjacent
        cases = [_with_literals(text, rng, rng.randint(0, 8)) for _ in range(200)]
        cases += ["<|endoftext|>", "<|endoftext|><|endoftext|>", "a<|im_start|>", "<|im_end|>b", "<|e<|end|>",
                  "<|endoftext", "\n\n<sep>\n\n<sep>", text[:100000] + "<|endoftext|>" + text[100000:150000]]
        for s in cases:
            d = s.encode()
            assert tok.encode(d).tolist() == encode_ex(d, table, pat, olits, ignore), repr(s[:200])
        # a batch of documents with literals
        docs = [c.encode() for c in cases[:150]]
        got = tok.encode_batch(docs)
        for d, g in zip(docs, got):
            assert g.tolist() == encode_ex(d, table, pat, olits, ignore)


def test_added_tokens_errors_and_unsupported_entry_points(gpu):
    import torch

    from paper_2607_29678_amd import Session, TokTierError

    m, vb, vo = stored_table(1)
    with _tok(m, vb, vo, "gpt2", False, [("<x>", 5000)]) as tok:
        with pytest.raises(TokTierError):
            tok.encode(b"ok<x>\x80")           # invalid UTF-8 after a literal
        with pytest.raises(TokTierError):
            tok.encode(b"\xc3<x>")             # a truncated character before one
        for call in (lambda: tok.encode_spans(b"a<x>"), lambda: tok.pretokenize(b"a<x>"), lambda: Session(tok)):
            with pytest.raises(TokTierError):
                call()
        d_in = torch.frombuffer(bytearray(b"a<x>b"), dtype=torch.uint8).cuda()
        d_out = torch.empty(8, dtype=torch.int32, device="cuda")
        d_len = torch.zeros(1, dtype=torch.int64, device="cuda")
        with pytest.raises(TokTierError):
            tok.encode_device(d_in, 5, d_out, d_len)
        assert tok.encode(b"<x>").tolist() == [5000]
        assert tok.encode(b"").tolist() == []
