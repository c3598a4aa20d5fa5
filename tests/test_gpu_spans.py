"""GPU parity of span export (IDs with byte and character spans) against the oracle.

Span i of the library is (byte begin, byte end, char begin, char end); the
oracle computes the same records from its IDs with the vocabulary's byte
lengths and a byte-to-character map (Appendix, Definition d:records; Route C,
span export).  Cases: the configuration texts (multi-byte characters split by
byte-level tokens in C4), long units whose tokens start many tiles before the
tile that encodes them, request lengths around tile edges and around
multiples of four, empty, tiny and invalid input, and the device entry point.
"""

import random

import numpy as np
import pytest

from conftest import config_bytes, lib_tokenizer, oracle_config_ids, oracle_ids, oracle_table, pattern_of
from oracle.spans import spans_of

pytestmark = pytest.mark.gpu

TILE_OWN = 1984


def _check(tok, k, data, want_ids=None, what=""):
    ids, spans = tok.encode_spans(data)
    table = oracle_table(k)
    if want_ids is None:
        want_ids = oracle_ids(data, table, pattern_of(k))
    assert ids.tolist() == list(want_ids), what
    want = spans_of(list(want_ids), data, table)
    got = [tuple(r) for r in spans.tolist()]
    if got != want:
        i = next(i for i in range(len(want)) if got[i] != want[i])
        raise AssertionError("%s: span %d of %d: got %s want %s" % (what, i, len(want), got[i], want[i]))


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_spans_config(gpu, k):
    _check(lib_tokenizer(k), k, config_bytes(k), oracle_config_ids(k), "config %d" % k)


@pytest.mark.parametrize("k", [1, 4])
def test_spans_long_units(gpu, k):
    """Units of up to 6,000 bytes: the tokens of an incoming unit start tiles before its encoder."""
    from test_gpu_long_units import _long_texts

    tok = lib_tokenizer(k)
    for i, data in enumerate(_long_texts(k, 55 + k)):
        _check(tok, k, data, what="long-unit case %d (%d bytes)" % (i, len(data)))


@pytest.mark.parametrize("k", [2, 4])
def test_spans_lengths(gpu, k):
    text = config_bytes(k)
    tok = lib_tokenizer(k)
    lengths = [1, 2, 3, 4, 5, 7, 8, 31, 32, 33, 64]
    lengths += [e * TILE_OWN + o for e in (1, 2, 3) for o in (-4, -3, -2, -1, 0, 1, 2, 3, 4)]
    for n in lengths:
        while n > 0 and (text[n] & 0xC0) == 0x80:  # cut at a character boundary
            n -= 1
        _check(tok, k, text[:n], what="length %d" % n)


def test_spans_multibyte_mix(gpu):
    rng = random.Random(5)
    alphabet = ["a", "é", "中", "\U0001F600", " ", "\n", "ж", "1", "'s", "文本"]
    tok = lib_tokenizer(4)
    for i in range(40):
        data = "".join(rng.choice(alphabet) for _ in range(rng.randint(1, 3000))).encode("utf-8")
        _check(tok, 4, data, what="mix %d" % i)


def test_spans_empty_and_invalid(gpu):
    tok = lib_tokenizer(1)
    ids, spans = tok.encode_spans(b"")
    assert ids.size == 0 and spans.shape == (0, 4)
    from paper_2607_29678_amd import TokTierError

    for bad in (b"\xff", b"ab\xc3", b"x" * 5000 + b"\xed\xa0\x80" + b"y" * 10):
        with pytest.raises(TokTierError):
            tok.encode_spans(bad)
    _check(tok, 1, b"ok after errors")


def test_spans_device_entry_point(gpu):
    torch = gpu
    k = 3
    data = config_bytes(k)[:300_000]
    tok = lib_tokenizer(k)
    want_ids, want_spans = tok.encode_spans(data)
    dev = torch.device("cuda:0")
    d_in = torch.from_numpy(np.frombuffer(data, dtype=np.uint8).copy()).to(dev)
    d_ids = torch.empty(len(data), dtype=torch.int32, device=dev)
    d_spans = torch.empty((len(data), 4), dtype=torch.int32, device=dev)
    d_len = torch.zeros(1, dtype=torch.int64, device=dev)
    s = torch.cuda.current_stream(dev)
    tok.encode_spans_device(d_in, len(data), d_ids, d_spans, d_len, s.cuda_stream)
    s.synchronize()
    T = int(d_len.item())
    assert T == want_ids.size
    assert np.array_equal(d_ids[:T].cpu().numpy(), want_ids)
    assert np.array_equal(d_spans[:T].cpu().numpy(), want_spans)
