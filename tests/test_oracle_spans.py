"""Pins of the oracle's token spans (CPU only).

The spans of byte-level BPE tokens follow from their IDs: byte offsets are a
running sum of token byte lengths, character spans come from the byte-to-char
map (Appendix, Definition d:records; Routes B and C, span export).  They are
pinned to:

  * a hand-worked request with a token that splits a two-byte character;
  * the offsets that the HF tokenizers library reports for the same merges with
    its byte-level pre-tokenizer (GPT-2 tables; library routine);
  * invariants on the configuration texts: byte spans partition the request and
    spell the tokens, and character spans cover exactly the characters those
    bytes belong to.
"""

import random

import pytest

from conftest import config_bytes, oracle_table, pattern_of, stored_table
from oracle.bpe import MergeTable
from oracle.spans import byte_to_char, encode_with_spans, spans_of
from test_oracle_bpe import _bytes_to_unicode


def test_hand_worked_split_character():
    # merges: (a, a) -> 256, (a, b) -> 257; no merge joins the two bytes of U+00E9
    vocab = [bytes([i]) for i in range(256)] + [b"aa", b"ab"]
    table = MergeTable([(97, 97, 256), (97, 98, 257)], vocab)
    data = "aé ab".encode("utf-8")  # a, e-acute (C3 A9), space, a, b
    ids, sp = encode_with_spans(data, table, "gpt2")
    assert ids == [97, 0xC3, 0xA9, 32, 257]
    assert sp == [(0, 1, 0, 1), (1, 2, 1, 2), (2, 3, 1, 2), (3, 4, 2, 3), (4, 6, 3, 5)]


def test_byte_to_char_map():
    assert byte_to_char("xé中\U0001F600".encode("utf-8")) == [0, 1, 1, 2, 2, 2, 3, 3, 3, 3, 4]
    assert byte_to_char(b"") == [0]


def _hf_tokenizer(k):
    tk = pytest.importorskip("tokenizers")
    m, _, _ = stored_table(k)
    t = oracle_table(k)
    b2u = _bytes_to_unicode()

    def s(tok):
        return "".join(b2u[x] for x in t.vocab[tok])

    strings = [s(i) for i in range(len(t.vocab))]
    if len(set(strings)) != len(strings):
        pytest.skip("table has duplicate byte strings; the HF model cannot represent it")
    tok = tk.Tokenizer(tk.models.BPE(vocab={st: i for i, st in enumerate(strings)},
                                     merges=[(s(a), s(b)) for a, b, _ in m.tolist()]))
    tok.pre_tokenizer = tk.pre_tokenizers.ByteLevel(add_prefix_space=False, use_regex=True)
    return tok


@pytest.mark.parametrize("k", [1, 2])
def test_char_spans_equal_hf_offsets(k):
    assert pattern_of(k) == "gpt2"
    hf = _hf_tokenizer(k)
    t = oracle_table(k)
    rng = random.Random(31 + k)
    alphabet = list("etaoin shrdlu\n\t'sS0123.,") + ["é", "ß", "中", "文", "\U0001F600", " ",
                                                        "́", "ж"]
    for _ in range(1500):
        text = "".join(rng.choice(alphabet) for _ in range(rng.randint(1, 30)))
        e = hf.encode(text)
        ids, sp = encode_with_spans(text.encode("utf-8"), t, "gpt2")
        assert e.ids == ids, text
        assert [tuple(o) for o in e.offsets] == [(c0, c1) for _, _, c0, c1 in sp], text


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_span_invariants_on_config_text(k):
    data = config_bytes(k)[:200_000]
    while data and (data[-1] & 0xC0) == 0x80:  # cut at a character boundary
        data = data[:-1]
    while data and data[-1] >= 0xC0:
        data = data[:-1]
    t = oracle_table(k)
    ids, sp = encode_with_spans(data, t, pattern_of(k))
    c = byte_to_char(data)
    text = data.decode("utf-8")
    prev_end = 0
    for tok, (b0, b1, c0, c1) in zip(ids, sp):
        assert b0 == prev_end and b1 > b0 and data[b0:b1] == t.vocab[tok]
        prev_end = b1
        # the character span holds exactly the characters the token's bytes belong to
        assert c0 == c[b0] and c1 == c[b1 - 1] + 1 and 0 <= c0 < c1 <= len(text)
        assert text[c0:c1].encode("utf-8").find(data[b0:b1]) >= 0
    assert prev_end == len(data)


def test_spans_reject_ids_that_do_not_spell_the_request():
    t = oracle_table(1)
    with pytest.raises(AssertionError):
        spans_of([ord("a")], b"ab", t)
