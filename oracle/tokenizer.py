"""Full-request tokenization, the definition the library must reproduce (oracle; test infrastructure).

The output contract (Sec. 1; Sec. 3 problem statement; Sec. 4.4 scope) is that
the IDs equal those of full reference tokenization of the whole request.  For
the tokenizers here that is: strict UTF-8 decoding, leftmost-first
pre-tokenization, per-piece BPE, concatenation (Appendix, Definition
d:frontend and Lemma l:homo).  A batch encodes each document on its own; no
piece or token crosses a document boundary (Sec. 4.2, multi-document batches).
"""

from .bpe import MergeTable, bpe
from .pretok import pretokenize


def decode_utf8(data: bytes) -> str:
    """Strict UTF-8 decoding; raises ``UnicodeDecodeError`` on invalid input."""
    return bytes(data).decode("utf-8", errors="strict")


def encode(data: bytes, table: MergeTable, pattern: str) -> list:
    """Token IDs of one request."""
    text = decode_utf8(data)
    out = []
    for a, b in pretokenize(text, pattern):
        out.extend(bpe(text[a:b].encode("utf-8"), table))
    return out


def encode_batch(docs, table: MergeTable, pattern: str) -> list:
    """Token IDs of each document of a batch."""
    return [encode(d, table, pattern) for d in docs]


def detokenize(ids, table: MergeTable) -> bytes:
    """Bytes spelled by a sequence of IDs."""
    return b"".join(table.vocab[i] for i in ids)
