"""GPU parity: the HIP library against the CPU oracle, split level and ID level.

The paper checks its GPU path at two levels, piece boundaries and final IDs,
because an ID-level comparison can hide a wrong split (Sec. 4.1).  Both are
compared element by element here on the seeded configurations, at their full
sizes, through the C ABI.
"""

import random

import numpy as np
import pytest

from conftest import config_bytes, lib_tokenizer, oracle_ids, oracle_table, pattern_of

pytestmark = pytest.mark.gpu



def _oracle_pieces(data: bytes, pattern: str):
    from oracle.pretok import piece_byte_starts

    return piece_byte_starts(data.decode("utf-8"), pattern)


def _oracle_config_ids(k):
    from conftest import oracle_config_ids

    return list(oracle_config_ids(k))


def _first_diff(a, b):
    n = min(len(a), len(b))
    for i in range(n):
        if a[i] != b[i]:
            return i
    return n if len(a) != len(b) else -1


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_split_parity_config(gpu, k):
    data = config_bytes(k)
    got = lib_tokenizer(k).pretokenize(data).tolist()
    want = _oracle_pieces(data, pattern_of(k))
    d = _first_diff(got, want)
    assert d == -1, "config %d: first piece difference at piece %d (lib %s, oracle %s)" % (
        k, d, got[d:d + 3], want[d:d + 3])


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_id_parity_config(gpu, k):
    got = lib_tokenizer(k).encode(config_bytes(k)).tolist()
    want = _oracle_config_ids(k)
    d = _first_diff(got, want)
    assert d == -1, "config %d: first ID difference at %d of %d/%d" % (k, d, len(got), len(want))


def test_batch_parity_c5(gpu):
    from workloads import textgen

    docs = [d.encode("utf-8") for d in textgen.batch_docs()]
    tok = lib_tokenizer(5)
    got = tok.encode_batch(docs)
    memo = {}
    for j, d in enumerate(docs):
        want = oracle_ids(d, oracle_table(5), "cl100k", memo)
        assert got[j].tolist() == want, "document %d" % j


def _fuzz_docs(seed, n_docs, alphabet, max_len):
    rng = random.Random(seed)
    return ["".join(rng.choice(alphabet) for _ in range(rng.randint(0, max_len))) for _ in range(n_docs)]


ALPHABET = list("asSltTrReEvVmMdD1 \n\t'.\r-_ ") + ["\u0085", " ", "ſ", "²", "中", "。",
                                                     "\U0001f600", "́", "　", "½", "А"]


@pytest.mark.parametrize("k", [1, 4])
def test_fuzz_batch_parity(gpu, k):
    """Thousands of short adversarial documents in one batch call, each against the oracle."""
    docs = _fuzz_docs(1000 + k, 4000, ALPHABET, 24)
    docs_b = [d.encode("utf-8") for d in docs]
    tok = lib_tokenizer(k)
    got = tok.encode_batch(docs_b)
    memo = {}
    for j, d in enumerate(docs_b):
        want = oracle_ids(d, oracle_table(k), pattern_of(k), memo)
        assert got[j].tolist() == want, "doc %d %r" % (j, docs[j])


@pytest.mark.parametrize("k", [1, 4])
def test_fuzz_split_parity(gpu, k):
    """Short adversarial strings one at a time through the split-level export."""
    tok = lib_tokenizer(k)
    for s in _fuzz_docs(2000 + k, 300, ALPHABET, 40):
        d = s.encode("utf-8")
        got = tok.pretokenize(d).tolist()
        want = _oracle_pieces(d, pattern_of(k))
        assert got == want, repr(s)


def test_empty_and_tiny(gpu):
    tok = lib_tokenizer(1)
    assert tok.encode(b"").tolist() == []
    for s in [b"a", b" ", b"\n", b"'", b"'s", b"1", b"\x00"]:
        assert tok.encode(s).tolist() == oracle_ids(s, oracle_table(1), "gpt2")


INVALID = [b"\x80", b"a\xc3", b"\xc3\x28", b"\xe0\x80\x80", b"\xed\xa0\x80", b"\xf4\x90\x80\x80",
           b"\xf8\x88\x80\x80\x80", b"\xc0\xaf", b"abc\xff", b"\xe2\x82", b"ok\xf0\x9f\x98"]


@pytest.mark.parametrize("bad", INVALID)
def test_invalid_utf8_is_error(gpu, bad):
    from paper_2607_29678_amd import TokTierError

    tok = lib_tokenizer(4)
    with pytest.raises(TokTierError) as e:
        tok.encode(bad)
    assert e.value.status == -5


def test_no_character_input_after_valid_call(gpu):
    """Regression: a request with no character at all (lone continuation bytes) has no piece; the
    output length must still be written, not left over from the previous call."""
    from paper_2607_29678_amd import TokTierError

    tok = lib_tokenizer(1)
    assert len(tok.encode(config_bytes(1))) > 100
    for bad in (b"\x80", b"\x80\x80\x80", b"\xbf" * 40):
        with pytest.raises(TokTierError) as e:
            tok.encode(bad)
        assert e.value.status == -5
    assert tok.encode(b"ok").tolist() == oracle_ids(b"ok", oracle_table(1), "gpt2")


def test_device_entry_matches_host(gpu):
    torch = gpu
    k = 3
    data = config_bytes(k)
    tok = lib_tokenizer(k)
    d_in = torch.from_numpy(np.frombuffer(data, dtype=np.uint8).copy()).cuda()
    d_out = torch.empty(len(data), dtype=torch.int32, device="cuda")
    d_len = torch.zeros(1, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream()
    tok.encode_device(d_in, len(data), d_out, d_len, stream.cuda_stream)
    stream.synchronize()
    T = int(d_len.item())
    assert d_out[:T].cpu().numpy().tolist() == _oracle_config_ids(k)


def test_stage_times_ring(gpu):
    """Stage events of the most recent calls are kept, oldest first, one entry per stage."""
    tok = lib_tokenizer(1)
    data = config_bytes(1)
    tok.set_profiling(3)
    try:
        for _ in range(5):
            tok.encode(data)
        calls = tok.stage_times()
    finally:
        tok.set_profiling(0)
    assert len(calls) == 3
    for c in calls:
        assert set(c) == {"tile"} and all(v > 0 for v in c.values())
