"""Pieces far longer than a tile under the walked patterns (o200k-style and
DeepSeek-style), against the oracle at split and ID level.

A piece of 64K characters covers about 33 tiles.  The tile it starts in walks
it once; every tile it covers takes it over from the previous tile's last
piece without walking it again, so the request costs one walk of the piece,
not one per tile.  The runs cover the alternatives that make long pieces:
lower-case and upper-case letter runs, an upper-case run with Lo letters and
marks inside (whose split depends on its last Lo letter), letters with marks,
whitespace with and without CR/LF, symbols, CJK/kana stretches, and digit
runs (pieces of three), with non-ASCII digits inside one of them.  The stress
request C5 is split under both patterns at full size too.
"""

import random
import time

import pytest

from conftest import oracle_ids, oracle_table, stored_table
from oracle.pretok import piece_byte_starts

pytestmark = pytest.mark.gpu

_TOK = {}


def _tok(pattern):
    from paper_2607_29678_amd import Tokenizer

    if pattern not in _TOK:
        m, vb, vo = stored_table(4)
        _TOK[pattern] = Tokenizer(m, vb, vo, pattern)
    return _TOK[pattern]


def _runs(rng, n):
    return {
        "lower": "".join(rng.choice("etaoinshrdlu") for _ in range(n)),
        "upper": "".join(rng.choice("ETAOINSHRDLU") for _ in range(n)),
        "upper_lo": "".join(rng.choice("ABCD") for _ in range(n - 3)) + "中" + "XY",
        "upper_lo_early": "中" + "".join(rng.choice("ABCD") for _ in range(n - 1)) + ".",
        "marks": "".join(rng.choice(["a", "́", "B", "̈"]) for _ in range(n)),
        "spaces": "".join(rng.choice(" \t") for _ in range(n)),
        "spaces_nl": "".join(rng.choice(" \t") for _ in range(n // 2)) + "\n" + " " * (n // 2),
        "symbols": "".join(rng.choice("-=*#") for _ in range(n)) + "\r\n/",
        "cjk": "".join(rng.choice("中文字漢語かなカナ") for _ in range(n)),
        "digits": "".join(rng.choice("0123456789") for _ in range(n)),
        "zeros": "0" * n,
        "digits_with_arabic_indic": "".join(rng.choice("0123456789") for _ in range(n // 2)) + "\u0663\u0664"
        + "".join(rng.choice("0123456789") for _ in range(n // 2)),
        "hyphens": "-" * n,
    }


@pytest.mark.parametrize("pattern", ["o200k", "deepseek"])
def test_runs_of_64k_characters(gpu, pattern):
    rng = random.Random(0x64 + len(pattern))
    tok = _tok(pattern)
    table = oracle_table(4)
    memo = {}  # the oracle's BPE of each distinct piece, shared by the two offsets
    for name, run in _runs(rng, 65_536).items():
        for off in (7, 1000):
            text = ("Ab. " * 300)[:1984 - off] + run + " tail Word."
            data = text.encode()
            starts = tok.pretokenize(data).tolist()
            ids = tok.encode(data).tolist()
            assert starts == piece_byte_starts(text, pattern), (pattern, name, off)
            assert ids == oracle_ids(data, table, pattern, memo), (pattern, name, off)
            # one walk of the piece per request, its part past the window read
            # 16 bytes at a time, and digit runs marked three bytes a step:
            # a warm call takes well under 20 ms (a character per step took
            # about 30 ms for these runs, a piece per step for digits more)
            t0 = time.perf_counter()
            tok.encode(data)
            dt = time.perf_counter() - t0
            assert dt < 0.02, (pattern, name, off, dt)


@pytest.mark.parametrize("pattern", ["o200k", "deepseek"])
def test_stress_request_split(gpu, pattern):
    from workloads import textgen

    text = textgen.config_text(5)
    data = text.encode("utf-8")
    tok = _tok(pattern)
    assert tok.pretokenize(data).tolist() == piece_byte_starts(text, pattern)
    tok.encode(data)
    t0 = time.perf_counter()
    tok.encode(data)
    dt = time.perf_counter() - t0
    assert dt < 0.05, (pattern, dt)  # (cl100k-style: about 1 ms)
