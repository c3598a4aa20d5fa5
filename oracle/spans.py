"""Token records with source spans (oracle; test infrastructure).

A token record is (id, a, b): the token's ID and the source span the offset
mapping reports for it (Appendix, Definition d:records).  For byte-level BPE
the byte length of every token is fixed by the vocabulary, so spans follow
from the IDs alone: a running sum of the tokens' byte lengths gives byte
offsets, and a byte-to-character map lifts those to character spans
(Appendix, Routes B and C, span export).

Definitions used here, for a request S of bytes B[0..n) whose IDs are
t_0 .. t_{T-1}:

  byte span of t_i:       [bb_i, be_i) with bb_0 = 0, be_i = bb_i + |vocab[t_i]|,
                          bb_{i+1} = be_i (the byte spans partition [0, n));
  char of byte p:         the index of the character whose encoding contains
                          byte p;
  character span of t_i:  [char(bb_i), char(be_i - 1) + 1).

A token that covers part of a multi-byte character therefore reports that
whole character, and several tokens of one character report the same span,
as the definition of records allows.
"""

from .bpe import MergeTable
from .tokenizer import decode_utf8, encode


def byte_to_char(data: bytes) -> list:
    """char(p) for every byte position p of a valid UTF-8 string, and char(n) = its length."""
    text = decode_utf8(data)
    out = []
    for ci, ch in enumerate(text):
        out.extend([ci] * len(ch.encode("utf-8")))
    out.append(len(text))
    assert len(out) == len(data) + 1
    return out


def spans_of(ids, data: bytes, table: MergeTable) -> list:
    """(byte_begin, byte_end, char_begin, char_end) of every token of `ids` over `data`."""
    c = byte_to_char(data)
    out = []
    p = 0
    for t in ids:
        q = p + len(table.vocab[t])
        out.append((p, q, c[p], c[q - 1] + 1))
        p = q
    assert p == len(data), "the tokens do not spell the request"
    return out


def encode_with_spans(data: bytes, table: MergeTable, pattern: str):
    """IDs of one request and the span of every token."""
    ids = encode(data, table, pattern)
    return ids, spans_of(ids, data, table)
