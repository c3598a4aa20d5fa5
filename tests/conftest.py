"""Shared fixtures: seeded texts, stored merge tables, oracle and library handles."""

import functools
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@functools.lru_cache(maxsize=None)
def stored_table(k):
    """(merges, vocab_bytes, vocab_offsets) of configuration k."""
    from workloads.tables import load_table

    return load_table(k)


@functools.lru_cache(maxsize=None)
def oracle_table(k):
    from oracle.bpe import MergeTable
    from workloads.tables import vocab_list

    m, vb, vo = stored_table(k)
    return MergeTable(m.tolist(), vocab_list(vb, vo))


@functools.lru_cache(maxsize=None)
def config_bytes(k):
    from workloads import textgen

    return textgen.config_text(k).encode("utf-8")


def pattern_of(k):
    from workloads import textgen

    return textgen.CONFIGS[k]["pattern"]


def oracle_ids(data: bytes, table, pattern: str, memo=None) -> list:
    """Oracle token IDs of one request; BPE results are memoised per distinct piece."""
    from oracle.bpe import bpe
    from oracle.pretok import pretokenize

    text = data.decode("utf-8")
    memo = {} if memo is None else memo
    out = []
    for a, b in pretokenize(text, pattern):
        piece = text[a:b].encode("utf-8")
        r = memo.get(piece)
        if r is None:
            r = memo[piece] = bpe(piece, table)
        out.extend(r)
    return out


@functools.lru_cache(maxsize=None)
def oracle_config_ids(k):
    """Oracle IDs of configuration k's full text (computed once per session)."""
    return tuple(oracle_ids(config_bytes(k), oracle_table(k), pattern_of(k)))


@pytest.fixture(scope="session")
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


_LIB_TOKS = {}


def lib_tokenizer(k):
    """Library handle of configuration k's table and pattern (cached)."""
    if k not in _LIB_TOKS:
        from paper_2607_29678_amd import Tokenizer

        m, vb, vo = stored_table(k)
        _LIB_TOKS[k] = Tokenizer(m, vb, vo, pattern_of(k))
    return _LIB_TOKS[k]
