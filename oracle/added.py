"""Added-token literals and ``ignore_merges`` (oracle; test infrastructure).

Two steps either side of BPE that production byte-level tokenizers use
(Sec. 4.2 and Sec. 4.5; Appendix, Definition d:frontend):

* Added tokens are literal strings the model reserves as single IDs.  The
  front end extracts them first with a leftmost-longest pass: scanning from the
  start, at every position the longest literal that matches there is taken
  and the scan resumes after it; a position where none matches is ordinary
  text.  The text between literals is then pre-tokenized and encoded segment
  by segment, with no piece crossing a literal (the units of the front end are
  the literals and the pieces of the segments).

* With ``ignore_merges`` the model stage first asks whether the whole piece is
  a vocabulary entry; if it is, the piece is that entry's single ID and no
  merge is applied.  Where several IDs spell the same bytes, the lowest ID is
  taken (reading: the paper does not say; a vocabulary keyed by its strings has
  one ID per string).

Both are written out plainly here on top of the oracle's pre-tokenizer and
BPE.
"""

from .bpe import MergeTable, bpe
from .pretok import pretokenize
from .tokenizer import decode_utf8


def vocab_index(table: MergeTable) -> dict:
    """bytes -> lowest ID spelling them."""
    idx = {}
    for i, v in enumerate(table.vocab):
        idx.setdefault(v, i)
    return idx


def split_added(data: bytes, literals) -> list:
    """Leftmost-longest extraction.  ``literals``: iterable of (bytes, id).
    Returns units in order: ("text", bytes) for the text between literals
    (never empty) and ("added", id) for every literal taken."""
    lits = [(bytes(b), int(i)) for b, i in literals]
    out = []
    text_start = 0
    p = 0
    n = len(data)
    while p < n:
        best = None
        for b, i in lits:
            if b and data.startswith(b, p) and (best is None or len(b) > len(best[0])):
                best = (b, i)
        if best is None:
            p += 1
            continue
        if p > text_start:
            out.append(("text", data[text_start:p]))
        out.append(("added", best[1]))
        p += len(best[0])
        text_start = p
    if n > text_start:
        out.append(("text", data[text_start:n]))
    return out


def encode_piece(piece: bytes, table: MergeTable, ignore_merges: bool, vidx=None) -> list:
    """IDs of one piece: the vocabulary entry itself under ignore_merges, else BPE."""
    if ignore_merges:
        vidx = vocab_index(table) if vidx is None else vidx
        hit = vidx.get(piece)
        if hit is not None:
            return [hit]
    return bpe(piece, table)


def encode_ex(data: bytes, table: MergeTable, pattern: str, literals=(), ignore_merges=False) -> list:
    """Token IDs of one request with added-token extraction and ignore_merges."""
    decode_utf8(data)  # the whole request must be strict UTF-8
    vidx = vocab_index(table) if ignore_merges else None
    out = []
    for kind, x in split_added(data, literals):
        if kind == "added":
            out.append(x)
            continue
        text = x.decode("utf-8")
        for a, b in pretokenize(text, pattern):
            out.extend(encode_piece(text[a:b].encode("utf-8"), table, ignore_merges, vidx))
    return out
