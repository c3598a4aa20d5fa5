"""The IDs of ``tt_encode`` through each delivery path, against the oracle.

A request in pageable host memory is encoded through pinned staging: when every
caller ID of the handle is below 65,536 the tile kernel writes the staged IDs
as 16-bit values, when below 2^24 as 16-bit values and their third bytes, and
the copy threads widen them into the caller's int32 array.  Pinned caller
buffers receive int32 IDs directly (the kernel's int32 stores, which staging
uses too for larger IDs).  All must give the oracle's IDs (Sec. 4.3 delivers
one request from host memory to host memory), at the full size of the
1,000,000-character GPT-2-style configuration and at a size below the copy
threads' split.
"""

import numpy as np
import pytest

from conftest import config_bytes, lib_tokenizer, oracle_config_ids, oracle_ids, oracle_table, stored_table

pytestmark = pytest.mark.gpu

K = 3        # GPT-2-style configuration: 50,000 merges, every ID below 65,536
SHIFT = 70_000  # moves every ID of the same table above 65,535 (24-bit staging)


def _shifted_handle():
    """The configuration's table with SHIFT distinct never-produced entries
    (invalid UTF-8) placed before its vocabulary, so that every ID grows by
    SHIFT."""
    from paper_2607_29678_amd import Tokenizer

    m, vb, vo = stored_table(K)
    idx = np.arange(SHIFT, dtype=np.uint32)
    dummy = np.empty((SHIFT, 5), dtype=np.uint8)
    dummy[:, 0] = 0xF8
    dummy[:, 1:] = idx.view(np.uint8).reshape(SHIFT, 4)
    vb2 = np.concatenate([dummy.reshape(-1), np.asarray(vb, dtype=np.uint8)])
    vo2 = np.concatenate([np.arange(SHIFT, dtype=np.int64) * 5, np.asarray(vo, dtype=np.int64) + 5 * SHIFT])
    m2 = np.asarray(m, dtype=np.int32) + SHIFT
    return Tokenizer(m2, vb2, vo2, "gpt2")


def _encode(tok, data_arr, out):
    n = tok.encode_into(data_arr, out)
    return np.asarray(out[:n], dtype=np.int64)


@pytest.mark.parametrize("size", ["full", "small"])
def test_staged_ids_all_paths(gpu, size):
    torch = gpu
    if size == "full":
        data = config_bytes(K)
        want = np.asarray(oracle_config_ids(K), dtype=np.int64)
    else:
        data = config_bytes(K).decode("utf-8")[:20_000].encode("utf-8")  # below the copy split
        want = np.asarray(oracle_ids(data, oracle_table(K), "gpt2"), dtype=np.int64)
    _, _, vo = stored_table(K)
    assert len(vo) - 1 <= 65536, "the configuration's IDs must fit in 16 bits"
    arr = np.frombuffer(data, dtype=np.uint8).copy()
    tok = lib_tokenizer(K)

    # pageable caller arrays: 16-bit staging, widened by the copy threads
    out = np.full(len(data), -7, dtype=np.int32)
    got = _encode(tok, arr, out)
    assert got.shape == want.shape and np.array_equal(got, want), "pageable (16-bit staging)"
    assert (out[len(want):] == -7).all(), "written past the IDs"

    # pinned caller buffers: int32 IDs straight into the caller's array
    pin_in = torch.from_numpy(arr).pin_memory()
    pin_out = torch.full((len(data),), -7, dtype=torch.int32).pin_memory()
    got = _encode(tok, pin_in, pin_out)
    assert np.array_equal(got, want), "pinned caller buffers"

    # the same table with IDs above 65,535: 24-bit staging
    tok2 = _shifted_handle()
    try:
        out2 = np.full(len(data), -7, dtype=np.int32)
        got2 = _encode(tok2, arr, out2)
        assert np.array_equal(got2 - SHIFT, want), "pageable (24-bit staging)"
        # and the 16-bit handle again after it (the staging is per handle and stream)
        got = _encode(tok, arr, out)
        assert np.array_equal(got, want), "pageable (16-bit staging), second call"
    finally:
        tok2.close()
