"""Pins of the trainer, the class table and the seeded inputs (CPU only)."""

import hashlib
import os

import numpy as np
import pytest

from conftest import stored_table
from oracle.classes import FOLDS, L, N, O, TABLE, W, char_class
from oracle.train import merge_word, train, train_from_counts, vocab_of
from workloads import textgen


# -- trainer -----------------------------------------------------------------

def test_hand_worked_corpus():
    # pieces "aaab" and "aab": pair counts (a,a)=3, (a,b)=2 -> first merge (a,a)
    merges = train_from_counts({b"aaab": 1, b"aab": 1}, 3)
    assert merges[0] == (97, 97, 256)
    # after it: "aaab" -> [aa, a, b], "aab" -> [aa, b]; counts (aa,a)=1,(a,b)=1,(aa,b)=1
    # -> ties broken by the smallest (left, right): (97, 98)
    assert merges[1] == (97, 98, 257)


def test_merge_word_leftmost_non_overlapping():
    assert merge_word([1, 1, 1, 1, 1], 1, 1, 9) == [9, 9, 1]
    assert merge_word([1, 2, 1, 2], 1, 2, 9) == [9, 9]


def test_trainer_deterministic_and_proper():
    text = textgen.training_text(1, 20_000)
    m1, v1 = train(text, "gpt2", 300)
    m2, v2 = train(text, "gpt2", 300)
    assert m1 == m2 and v1 == v2
    seen = set(range(256))
    for r, (a, b, c) in enumerate(m1):
        assert a in seen and b in seen and c == 256 + r
        seen.add(c)
        assert v1[c] == v1[a] + v1[b]


@pytest.mark.parametrize("k,want", [
    (1, "fc21a7b7a72bea2099526bbacc1b2d719831d02b597f77246ab4754118e6f80e"),
    (2, "a902abe49feb96bbe47ad0837182a12234795e4a12051b14af896bfe18d14796"),
    (3, "4d63a2a1b3e2fe1d43bdb36949ca77ed2726471b7a114ec96181c6ed709d2ab7"),
    (4, "b961e8970a8fdc39aaa5439646c3eba292f942bd96d01942cd8b3b7e913e83c8"),
])
def test_stored_tables_pinned_and_proper(k, want):
    m, vb, vo = stored_table(k)
    assert hashlib.sha256(m.astype(np.int32).tobytes()).hexdigest() == want
    assert len(m) == textgen.CONFIGS[k]["merges"]
    from workloads.tables import vocab_list

    vocab = vocab_list(vb, vo)
    assert vocab == vocab_of([tuple(x) for x in m.tolist()])


def test_stored_table_c1_retrains_identically():
    m, _, _ = stored_table(1)
    merges, _ = train(textgen.training_text(1), "gpt2", 1024)
    assert merges == [tuple(x) for x in m.tolist()]


# -- class table ---------------------------------------------------------------

WHITE_SPACE = [0x09, 0x0A, 0x0B, 0x0C, 0x0D, 0x20, 0x85, 0xA0, 0x1680] + list(range(0x2000, 0x200B)) + \
              [0x2028, 0x2029, 0x202F, 0x205F, 0x3000]


def test_whitespace_is_unicode_white_space():
    assert sorted(c for c in range(0x110000) if TABLE[c] == W) == WHITE_SPACE


@pytest.mark.parametrize("cp,cls", [(ord("A"), L), (ord("z"), L), (ord("5"), N), (0xB2, N), (0xBD, N),
                                    (0x2163, N), (0x4E2D, L), (0x3002, O), (0x301, O), (0x1F600, O),
                                    (0x1C, O), (0x1F, O), (0x17F, L), (0x410, L), (0x5F, O)])
def test_class_spot_checks(cp, cls):
    assert char_class(cp) == cls


def test_contraction_folds():
    assert FOLDS["s"] == frozenset([0x53, 0x73, 0x17F])
    for ch in "trevmld":
        assert FOLDS[ch] == frozenset([ord(ch), ord(ch.upper())])


@pytest.mark.slow
def test_class_table_equals_fresh_engine_probe():
    tk = pytest.importorskip("tokenizers")
    cps = [c for c in range(0x110000) if not 0xD800 <= c <= 0xDFFF]
    text = "".join(map(chr, cps))
    for code, pat in ((L, r"\p{L}"), (N, r"\p{N}"), (W, r"\s")):
        sp = tk.pre_tokenizers.Split(tk.Regex(pat), behavior="removed")
        left = bytearray(len(cps))
        for _, (a, b) in sp.pre_tokenize_str(text):
            left[a:b] = b"\x01" * (b - a)
        members = {cps[i] for i in range(len(cps)) if not left[i]}
        assert members == {c for c in range(0x110000) if TABLE[c] == code}


def test_class_table_file_pinned():
    from oracle.classes import TABLE_PATH

    with open(TABLE_PATH, "rb") as f:
        assert hashlib.sha256(f.read()).hexdigest() == \
            "316e731861e64a3ef93bf357e77bcf74fb590852d0654deb2869f91f4d3628e1"


def test_o200k_class_table_file_pinned():
    from oracle.classes import O200K_PATH

    with open(O200K_PATH, "rb") as f:
        assert hashlib.sha256(f.read()).hexdigest() == \
            "6abc8e629552010cc1dcd36fc4a5e1304673a577c290d061a62ba04536c394e4"


@pytest.mark.slow
@pytest.mark.parametrize("code,pats", [("UP", (r"\p{Lu}", r"\p{Lt}")), ("LO", (r"\p{Ll}",)),
                                       ("BO", (r"\p{Lm}", r"\p{Lo}")), ("MK", (r"\p{M}",))])
def test_o200k_class_table_equals_fresh_engine_probe(code, pats):
    tk = pytest.importorskip("tokenizers")
    from oracle.classes import BO, LO, MK, O200K_TABLE, UP

    cps = [c for c in range(0x110000) if not 0xD800 <= c <= 0xDFFF]
    text = "".join(map(chr, cps))
    members = set()
    for pat in pats:
        sp = tk.pre_tokenizers.Split(tk.Regex(pat), behavior="removed")
        left = bytearray(len(cps))
        for _, (a, b) in sp.pre_tokenize_str(text):
            left[a:b] = b"\x01" * (b - a)
        members |= {cps[i] for i in range(len(cps)) if not left[i]}
    want = {"UP": UP, "LO": LO, "BO": BO, "MK": MK}[code]
    assert members == {c for c in range(0x110000) if O200K_TABLE[c] == want}


def test_o200k_classes_spot_checks():
    from oracle.classes import BO, LO, MK, N, O, UP, W, o200k_class

    assert [o200k_class(ord(c)) for c in "Aaǅ中ʰ\u03011 ./"] == [UP, LO, UP, BO, BO, MK, N, W, O, O]


# -- seeded inputs --------------------------------------------------------------

@pytest.mark.parametrize("k,chars,nbytes", [
    (1, 10_000, 10_000),
    (2, 100_000, 100_000),
    (3, 1_000_000, 1_000_000),
    (4, 1_000_000, 1_286_791),
    (5, 3_000_000, 3_771_319),
])
def test_config_sizes(k, chars, nbytes):
    from conftest import config_bytes

    b = config_bytes(k)
    assert len(b) == nbytes
    assert len(b.decode("utf-8")) == chars


def test_config_texts_pinned():
    from conftest import config_bytes

    got = {k: hashlib.sha256(config_bytes(k)).hexdigest()[:16] for k in (1, 2, 3, 4, 5)}
    assert got == PINNED_TEXT_SHA


PINNED_TEXT_SHA = {1: '2c0a608010eb6915', 2: 'dc4df0b25ae13a4b', 3: '0614ca4159d1ba93',
                   4: '5e70667c701ff553', 5: '03715c15f73d1bd9'}


def test_c1_shares():
    from conftest import config_bytes

    s = config_bytes(1).decode()
    assert abs(sum(c.isdigit() for c in s) / len(s) - 0.05) <= 0.01
    assert abs(sum(c in ",;:()\"-'.?!" for c in s) / len(s) - 0.05) <= 0.01
    assert all(ord(c) < 128 for c in s)


def test_c4_multibyte_share():
    from conftest import config_bytes

    s = config_bytes(4).decode()
    assert abs(sum(ord(c) > 127 for c in s) / len(s) - 0.20) <= 0.01


def test_c5_stress_runs_present():
    from conftest import config_bytes

    s = config_bytes(5).decode()
    for run in ("a" * 25_000, "-" * 25_000, "=" * 25_000, "0" * 25_000):
        assert run in s
    docs = textgen.batch_docs()
    assert len(docs) == 64 and all(len(d) == 16_384 for d in docs)
