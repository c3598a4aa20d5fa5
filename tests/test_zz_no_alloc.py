"""The entry point that allocates nothing (``tt_encode_device_noalloc``) against
``tt_encode_device`` on the same handle and inputs: identical IDs and lengths,
on two calls in a row with the second one smaller (the fixed workspace keeps
the first call's words), on the GPT-2-style and cl100k-style tables, and at
the size limit.  Also its host-side rejections, which enqueue nothing."""

import ctypes

import numpy as np
import pytest

from conftest import config_bytes, pattern_of, stored_table

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _cut(data, n):
    """The first n bytes of data, moved back to a character boundary."""
    n = min(n, len(data))
    while 0 < n < len(data) and (data[n] & 0xC0) == 0x80:
        n -= 1
    return data[:n]


def _run(tok, fn, data, stream):
    dev = torch.device("cuda:0")
    d_in = torch.from_numpy(np.frombuffer(data, dtype=np.uint8).copy()).to(dev)
    d_out = torch.full((max(1, len(data)),), -7, dtype=torch.int32, device=dev)
    d_len = torch.full((1,), -99, dtype=torch.int64, device=dev)
    getattr(tok, fn)(d_in, len(data), d_out, d_len, stream.cuda_stream)
    stream.synchronize()
    n = int(d_len.item())
    return n, d_out[: max(n, 0)].cpu().numpy()


@pytest.mark.parametrize("k", [3, 4])
def test_noalloc_equals_device_entry_point(k):
    from paper_2607_29678_amd import Tokenizer

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream(0)
    m, vb, vo = stored_table(k)
    text = config_bytes(k)
    first = _cut(text, 1_200_000)
    second = _cut(first, 123_457)  # smaller, and inside the first call's range
    with Tokenizer(m, vb, vo, pattern_of(k)) as tok:
        for data in (first, second, _cut(first, 5000), b"x"):
            n_ref, ids_ref = _run(tok, "encode_device", data, stream)
            n, ids = _run(tok, "encode_device_noalloc", data, stream)
            assert n_ref > 0 and n == n_ref
            assert np.array_equal(ids, ids_ref)


def test_noalloc_at_the_limit_and_beyond():
    from paper_2607_29678_amd import Tokenizer, _lib

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream(0)
    m, vb, vo = stored_table(3)
    text = config_bytes(3)  # ASCII: any cut is a character boundary
    big = (text * (_lib.TT_NOALLOC_MAX_BYTES // len(text) + 1))[: _lib.TT_NOALLOC_MAX_BYTES]
    with Tokenizer(m, vb, vo, "gpt2") as tok:
        n_ref, ids_ref = _run(tok, "encode_device", big, stream)
        n, ids = _run(tok, "encode_device_noalloc", big, stream)
        assert n == n_ref and np.array_equal(ids, ids_ref)
        # one byte more is rejected on the host, before anything is enqueued
        lib = tok._lib
        d_len = torch.zeros(1, dtype=torch.int64, device="cuda:0")
        st = lib.tt_encode_device_noalloc(tok._h, ctypes.c_void_p(1), _lib.TT_NOALLOC_MAX_BYTES + 1,
                                          ctypes.c_void_p(1), ctypes.c_void_p(d_len.data_ptr()),
                                          ctypes.c_void_p(stream.cuda_stream))
        assert st == -6  # TT_ERR_TOO_LARGE
        # the empty request writes a zero length
        d_len.fill_(5)
        st = lib.tt_encode_device_noalloc(tok._h, None, 0, None, ctypes.c_void_p(d_len.data_ptr()),
                                          ctypes.c_void_p(stream.cuda_stream))
        stream.synchronize()
        assert st == 0 and int(d_len.item()) == 0
        # invalid input: the error code in the length word, as for tt_encode_device
        n, _ = _run(tok, "encode_device_noalloc", b"ab\xc3(", stream)
        assert n == -5
