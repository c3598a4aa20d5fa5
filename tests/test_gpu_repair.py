"""Incremental repair on the GPU: sessions against the oracle.

After every append the session's records must equal the oracle's full
tokenization of the whole text, IDs and spans (the output contract of
Sec. 3.2: repair may do more work, never produce different IDs).  The tokens
before `kept` must be exactly those of the previous sequence.
"""

import random

import numpy as np
import pytest

from conftest import lib_tokenizer, oracle_table, pattern_of
from oracle.spans import encode_with_spans

pytestmark = pytest.mark.gpu


def _session(k, window=0):
    from paper_2607_29678_amd import Session

    return Session(lib_tokenizer(k), window)


def _check(sess, text: str, k, prev_ids=None, info=None):
    ids, spans = sess.tokens()
    want_ids, want_spans = encode_with_spans(text.encode("utf-8"), oracle_table(k), pattern_of(k))
    assert ids.tolist() == want_ids
    assert [tuple(s) for s in spans.tolist()] == [tuple(s) for s in want_spans]
    if prev_ids is not None and info is not None:
        assert info["n_tokens"] == len(want_ids)
        assert ids[: info["kept"]].tolist() == prev_ids[: info["kept"]].tolist()
    return ids


@pytest.mark.parametrize("k", [1, 2, 4])
def test_session_random_appends(gpu, k):
    """A seeded text appended in random chunks of 1..600 characters."""
    from workloads import textgen

    text = textgen.config_text(k)[:40000]
    rng = random.Random(0xA99E + k)
    sess = _session(k)
    pos, ids = 0, np.zeros(0, dtype=np.int32)
    windows = []
    while pos < len(text):
        step = rng.choice([1, 2, 5, 30, 200, 600]) if pos else 3000
        nxt = min(len(text), pos + rng.randint(1, step))
        info = sess.append(text[pos:nxt].encode("utf-8"))
        pos = nxt
        ids = _check(sess, text[:pos], k, ids, info)
        windows.append(info["windows"])
    assert sess.info()["chars"] == len(text)
    # natural text: the first window is admitted almost always
    assert sum(1 for w in windows[1:] if w == 1) >= 0.9 * (len(windows) - 1)


@pytest.mark.parametrize("k", [1, 4])
def test_session_adversarial_appends(gpu, k):
    """Appends that move boundaries far back; long same-class runs force
    wider windows and, past the widest, the whole-text fallback."""
    # expected route: "fallback" (six windows rejected, then the whole text),
    # "window" (a window admitted), None (either; exactness is what matters)
    cases = [
        ("x " + "1" * 20000, "1", "fallback"),    # no boundary inside 16K characters of digits
        ("abc" + " " * 20000, "d", "fallback"),   # one whitespace run
        ("q." + "\n" * 3000, "\n z", None),       # windows inside the run, then one reaching the start
        ("lorem ipsum " * 300 + " pipe", "line", "window"),
        ("text " * 300 + "don", "'t", "window"),
        ("é" * 100 + "中文" * 500, "。x", None),   # one letter run of 1,100 characters
    ]
    for a, b, route in cases:
        sess = _session(k)
        sess.append(a.encode())
        prev = _check(sess, a, k)
        info = sess.append(b.encode())
        _check(sess, a + b, k, prev, info)
        if route == "fallback":
            assert info["full"] == 1 and info["windows"] == 6, info
        elif route == "window":
            assert info["full"] == 0, info


def test_session_window_widths(gpu):
    """Small first windows widen; every width gives the same IDs."""
    from workloads import textgen

    text = textgen.config_text(2)[:20000]
    for w in (4, 32, 512, 4096):
        sess = _session(2, w)
        rng = random.Random(w)
        pos, ids = 0, np.zeros(0, dtype=np.int32)
        while pos < len(text):
            nxt = min(len(text), pos + rng.randint(1, 2500))
            info = sess.append(text[pos:nxt].encode())
            pos = nxt
            ids = _check(sess, text[:pos], 2, ids, info)


def test_session_empty_invalid_and_multibyte(gpu):
    from paper_2607_29678_amd import TokTierError

    sess = _session(4)
    info = sess.append(b"")
    assert info["n_tokens"] == 0 and sess.info()["bytes"] == 0
    sess.append("Ünïcode tëxt ".encode() * 50)
    before = sess.tokens()[0].copy()
    state = sess.info()
    for bad in (b"\x80abc", b"ok\xc3", b"\xed\xa0\x80"):
        with pytest.raises(TokTierError):
            sess.append(bad)
        assert sess.info() == state
        assert sess.tokens()[0].tolist() == before.tolist()
    text = "Ünïcode tëxt " * 50
    for piece in ["中", "文。", "😀", " ſ's", "\r\n", "123", "4567"]:
        info = sess.append(piece.encode())
        text += piece
        before = _check(sess, text, 4, before, info)
    assert sess.info()["chars"] == len(text)


def test_session_large_context(gpu):
    """A 1,000,000-character session (the transcript workload) with appends of
    about 1,500 characters."""
    from workloads import textgen

    text = textgen.latency_sample(3, 0)
    extra = textgen.latency_sample(3, 1)[:12000]
    sess = _session(3)
    sess.append(text.encode())
    ids = _check(sess, text, 3)
    rng = random.Random(3)
    pos = 0
    while pos < len(extra):
        nxt = min(len(extra), pos + rng.randint(800, 2500))
        info = sess.append(extra[pos:nxt].encode())
        pos = nxt
        ids = _check(sess, text + extra[:pos], 3, ids, info)
        assert info["full"] == 0 and info["windows"] == 1
