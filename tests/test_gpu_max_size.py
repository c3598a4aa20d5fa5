"""Requests of the largest accepted size (TT_MAX_BYTES = 2^30 bytes) on the GPU.

The oracle cannot tokenize a gigabyte in a test, so the request is built to
have a property that holds at any size: it is a block B of seeded text
repeated k times, followed by copies of two tiny blocks P1 and P2 that bring
the length to exactly 2^30.  Every block starts with an ASCII capital letter
and ends with ".\\n".  Each pattern's decisions at a position depend on a few
characters around it, the same at every junction, so no piece crosses a
junction and every block is split and merged as it is on its own: the IDs of
the request are the blocks' oracle IDs, concatenated.  The test checks this
on a short request with every kind of junction (B|B, B|P1, P1|P1, P1|P2,
P2|P2 and the end of the text) with the oracle, then compares the GPU's
output over the whole gigabyte element by element.

The tile edges (every 1,984 bytes) fall at every offset of B, since B's
length is not a multiple of the tile size.  One byte more than the maximum
is an error (TT_ERR_TOO_LARGE) that the library raises before any work.
"""

import re

import numpy as np
import pytest

from conftest import config_bytes, oracle_ids, oracle_table, pattern_of, stored_table

pytestmark = pytest.mark.gpu

MAX_BYTES = 1 << 30
P1 = b"A.\n"
P2 = b"Ab.\n"


def _block(k, min_len):
    """A piece of configuration k's text that starts with a capital after ".\\n" and ends with
    ".\\n" before a capital, at least ``min_len`` bytes long."""
    text = config_bytes(k).decode("utf-8")
    starts = [m.start() + 2 for m in re.finditer(r"\.\n[A-Z]", text)]
    i = starts[0]
    j = next(s for s in starts if len(text[i:s].encode("utf-8")) >= min_len)
    return text[i:j].encode("utf-8")


def _fill(block_len):
    """(k, a, b) with k * block_len + 3 a + 4 b == MAX_BYTES."""
    k = (MAX_BYTES - 64) // block_len
    r = MAX_BYTES - k * block_len
    for b in range(3):
        if (r - 4 * b) % 3 == 0:
            return k, (r - 4 * b) // 3, b
    raise AssertionError("no filler")


@pytest.mark.parametrize("k", [3, 4])
def test_max_size_request(gpu, k):
    from paper_2607_29678_amd import TokTierError, Tokenizer

    table, pat = oracle_table(k), pattern_of(k)
    block = _block(k, 60000)
    reps, a, b = _fill(len(block))
    assert reps * len(block) + 3 * a + 4 * b == MAX_BYTES and reps > 10000
    memo = {}
    ib, i1, i2 = (oracle_ids(x, table, pat, memo) for x in (block, P1, P2))
    # the junctions, at the oracle level
    short = block * 2 + P1 * 2 + P2 * 2
    assert oracle_ids(short, table, pat, memo) == ib * 2 + i1 * 2 + i2 * 2
    want = np.concatenate([np.tile(np.asarray(ib, np.int32), reps), np.tile(np.asarray(i1, np.int32), a),
                           np.tile(np.asarray(i2, np.int32), b)])
    data = block * reps + P1 * a + P2 * b
    assert len(data) == MAX_BYTES
    m, vb, vo = stored_table(k)
    tok = Tokenizer(m, vb, vo, pat)
    try:
        got = tok.encode(data)
        assert got.shape == want.shape, (got.shape, want.shape)
        bad = np.flatnonzero(got != want)
        assert bad.size == 0, "first difference at ID %d of %d" % (bad[0], want.size)
        with pytest.raises(TokTierError) as e:
            tok.encode(data + b"A")
        assert e.value.status == -6
    finally:
        tok.close()
