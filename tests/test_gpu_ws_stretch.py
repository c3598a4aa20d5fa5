"""cl100k-style rule for whitespace after CR/LF, when the stretch runs far past
the tile's window.

After CR/LF, a whitespace stretch is a piece of its own (``\\s+(?!\\S)``) or
joins the CR/LF (``\\s*[\\r\\n]+``) depending on what ends it: more CR/LF, or
something else.  When the stretch reaches past the 2,048-byte window, the tile
reads on in global memory with one wave (16 bytes per lane per step) until the
stretch ends.  The cases: stretches of about 70,000 bytes (some 35 tiles) that
end in CR/LF, in a letter, at the end of the text, at a document end inside a
batch, with non-ASCII whitespace (U+3000, U+00A0, U+2028) and tabs, vertical
tabs and form feeds inside, and at several offsets from a tile edge.  Split
and ID parity against the oracle; every request must take well under a second
(one character per step in global memory took milliseconds per request).
"""

import time

import pytest

from conftest import lib_tokenizer, oracle_ids, oracle_table
from oracle.pretok import piece_byte_starts

pytestmark = pytest.mark.gpu

K = 4  # cl100k-style pattern


def _cases():
    sp = " " * 70_000
    mix = "".join(" \t\x0b\x0c"[i % 4] for i in range(70_000))
    return {
        "then_crlf": "ab\n" + sp + "\r\nxy",
        "then_letter": "ab\n" + sp + "xy",
        "to_text_end": "ab\n" + sp,
        "mixed_then_lf": "ab\r\n" + mix + "\n",
        "mixed_then_letter": "ab\r\n" + mix + "q",
        "ideographic_inside_then_lf": "ab\n" + sp[:30_000] + "\u3000" + sp[:30_000] + "\nz",
        "nbsp_inside_then_letter": "ab\n" + sp[:30_000] + "\u00a0" + sp[:30_000] + "z",
        "line_sep_at_end": "ab\n" + sp[:40_000] + "\u2028",
        "two_stretches": "ab\n" + sp[:5_000] + "\n" + sp + "\nc",
    }


@pytest.mark.parametrize("name", sorted(_cases()))
def test_long_stretch_after_crlf(gpu, name):
    tok = lib_tokenizer(K)
    table = oracle_table(K)
    base = _cases()[name]
    for off in (0, 5, 1977, 1990):
        text = ("Word, " * 700)[:off] + base
        data = text.encode("utf-8")
        t0 = time.perf_counter()
        starts = tok.pretokenize(data).tolist()
        ids = tok.encode(data).tolist()
        dt = time.perf_counter() - t0
        assert starts == piece_byte_starts(text, "cl100k"), (name, off)
        assert ids == oracle_ids(data, table, "cl100k"), (name, off)
        assert dt < 1.0, (name, off, dt)


def test_long_stretch_to_document_end_in_batch(gpu):
    tok = lib_tokenizer(K)
    table = oracle_table(K)
    docs = [("x\n" + " " * 70_000).encode(), ("   \n b").encode(), ("y\r\n" + " " * 9_000 + "\n").encode(),
            ("z" * 3).encode()]
    got = tok.encode_batch(docs)
    for j, d in enumerate(docs):
        assert got[j].tolist() == oracle_ids(d, table, "cl100k"), "document %d" % j


@pytest.mark.parametrize("tail", ["\r\nxy", "xy"])
def test_long_stretch_deep_in_a_large_request(gpu, tail):
    """A 150,000-byte stretch after CR/LF that starts 300,000 bytes into a
    pageable request of more than 256 KB (staged through pinned memory by the
    copy threads), so that the read past the window starts far from the
    request's first tiles."""
    tok = lib_tokenizer(K)
    table = oracle_table(K)
    text = ("Word, " * 50_000) + "ab\n" + " " * 150_000 + tail + " more words" * 1000
    data = text.encode("utf-8")
    assert len(data) > 256 * 1024
    ids = tok.encode(data).tolist()
    assert ids == oracle_ids(data, table, "cl100k")
    assert tok.pretokenize(data).tolist() == piece_byte_starts(text, "cl100k")
