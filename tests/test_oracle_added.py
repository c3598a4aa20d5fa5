"""Oracle pins for added-token literals and ignore_merges.

* Hand-worked leftmost-longest extractions and a hand-built merge list on
  which ignore_merges changes the result.
* Library routine: HF tokenizers 0.22.2 (the paper's pinned reference) built
  from the same merges, with the pattern as a Split pre-tokenizer, the
  byte-level alphabet, the literals as added tokens and the BPE model's
  ignore_merges option, agrees with the oracle on seeded text with literals
  inserted (including overlapping and nested literals).
"""

import random

import pytest

from conftest import oracle_table, stored_table
from oracle.added import encode_ex, split_added, vocab_index
from oracle.bpe import MergeTable, bpe
from test_oracle_bpe import _bytes_to_unicode
from test_oracle_pretok import REGEX


@pytest.mark.parametrize("data,lits,want", [
    (b"x<a>bc", [(b"<a>", 1), (b"<a>b", 2)], [("text", b"x"), ("added", 2), ("text", b"c")]),
    (b"abc", [(b"ab", 1), (b"bc", 2)], [("added", 1), ("text", b"c")]),          # leftmost wins
    (b"abc", [(b"bc", 2), (b"abc", 3), (b"ab", 1)], [("added", 3)]),            # then longest
    (b"aaaa", [(b"aa", 7)], [("added", 7), ("added", 7)]),
    (b"aaa", [(b"aa", 7)], [("added", 7), ("text", b"a")]),
    (b"<|e|><|e|>", [(b"<|e|>", 5)], [("added", 5), ("added", 5)]),
    ("é<é>é".encode(), [("<é>".encode(), 9)], [("text", "é".encode()), ("added", 9), ("text", "é".encode())]),
    (b"plain", [(b"<x>", 1)], [("text", b"plain")]),
    (b"", [(b"<x>", 1)], []),
])
def test_leftmost_longest_hand_worked(data, lits, want):
    assert split_added(data, lits) == want


def _abc_table():
    """Merges r0 (b,c), r1 (a,b), r2 (ab,c): BPE("abc") merges (b,c) first and
    ends as [a, bc], although "abc" is itself a vocabulary entry."""
    vocab = [bytes([i]) for i in range(256)] + [b"bc", b"ab", b"abc"]
    a, b, c = ord("a"), ord("b"), ord("c")
    merges = [(b, c, 256), (a, b, 257), (257, c, 258)]
    return MergeTable(merges, vocab)


def test_ignore_merges_hand_worked():
    t = _abc_table()
    assert bpe(b"abc", t) == [ord("a"), 256]
    assert encode_ex(b"abc", t, "gpt2", ignore_merges=True) == [258]
    assert encode_ex(b"abc", t, "gpt2", ignore_merges=False) == [ord("a"), 256]
    # pieces, not the whole text: " abc" is one GPT-2 piece that is no entry
    assert encode_ex(b"x abc", t, "gpt2", ignore_merges=True) == [ord("x")] + bpe(b" abc", t)
    # the lowest ID among duplicate spellings
    t2 = MergeTable(t.merges, t.vocab + [b"abc"])
    assert vocab_index(t2)[b"abc"] == 258


def _hf_tokenizer(k, pattern, literals, ignore_merges):
    tk = pytest.importorskip("tokenizers")
    m, _, _ = stored_table(k)
    t = oracle_table(k)
    b2u = _bytes_to_unicode()

    def s(tok):
        return "".join(b2u[x] for x in t.vocab[tok])

    strings = [s(i) for i in range(len(t.vocab))]
    assert len(set(strings)) == len(strings)
    model = tk.models.BPE(vocab={st: i for i, st in enumerate(strings)},
                          merges=[(s(a), s(b)) for a, b, _ in m.tolist()], ignore_merges=ignore_merges)
    tok = tk.Tokenizer(model)
    tok.pre_tokenizer = tk.pre_tokenizers.Sequence([
        tk.pre_tokenizers.Split(tk.Regex(REGEX[pattern]), behavior="isolated"),
        tk.pre_tokenizers.ByteLevel(add_prefix_space=False, use_regex=False),
    ])
    tok.add_special_tokens([tk.AddedToken(x, special=True, normalized=False) for x in literals])
    return tok, {x.encode(): tok.token_to_id(x) for x in literals}


LITERALS = ["<|endoftext|>", "<|im_start|>", "<|im_end|>", "<|e", "<|end", "[INST]", "é<é>", "\n\n<sep>"]


@pytest.mark.parametrize("k,pattern", [(1, "gpt2"), (4, "cl100k")])
@pytest.mark.parametrize("ignore_merges", [False, True])
def test_against_hf_tokenizers(k, pattern, ignore_merges):
    from workloads import textgen

    tok, lit_ids = _hf_tokenizer(k, pattern, LITERALS, ignore_merges)
    table = oracle_table(k)
    base = textgen.config_text(k)
    rng = random.Random(31 * k + ignore_merges)
    for _ in range(300):
        a = rng.randint(0, len(base) - 400)
        parts = []
        for _ in range(rng.randint(0, 6)):
            parts.append(base[a:a + rng.randint(0, 60)])
            a += 60
            parts.append(rng.choice(LITERALS + ["<|", "|>", "<|im_", "é<", "<é>"]))
        parts.append(base[a:a + rng.randint(0, 60)])
        text = "".join(parts)
        want = tok.encode(text, add_special_tokens=False).ids
        got = encode_ex(text.encode(), table, pattern, literals=list(lit_ids.items()), ignore_merges=ignore_merges)
        assert got == want, repr(text)


@pytest.mark.parametrize("k,pattern", [(1, "gpt2"), (4, "cl100k")])
def test_ignore_merges_changes_some_pieces(k, pattern):
    """On the stored tables, whole-piece probes and BPE agree on most pieces
    (trained merges rebuild their own words); the test records that the two
    paths are exercised, and that they agree with HF on both sides."""
    from oracle.pretok import pretokenize
    from workloads import textgen

    table = oracle_table(k)
    vidx = vocab_index(table)
    text = textgen.config_text(k)[:20000]
    hits = sum(1 for a, b in pretokenize(text, pattern) if text[a:b].encode() in vidx)
    assert hits > 1000
