"""Exact GPU tokenization for AMD Instinct MI355X (gfx950).

A HIP library (``libtoktier.so``, C ABI in ``include/toktier.h``) that computes
the full-request tokenization path of TokTier: GPT-family pre-tokenization
recast as run-local rules, then exact byte-level BPE and output compaction,
with token IDs identical to full reference tokenization.  This package holds
the library sources (``csrc/``), its build script and a thin ctypes binding.
"""

from .tokenizer import (CL100K, DEEPSEEK, GPT2, O200K, PATTERNS, Session, Tokenizer, splice_plan,  # noqa: F401
                        status_string, sync_boundaries)
from ._lib import TokTierError  # noqa: F401


def build(verbose: bool = False) -> str:
    from ._build import build as _b

    return _b(verbose)
