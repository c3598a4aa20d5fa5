"""Seeded synthetic inputs for the tokenizer.

This package only produces text and loads stored merge tables.  It holds none
of the tokenizer's arithmetic (no matching, no merging): both the CPU oracle
and the HIP library consume what it produces.
"""

from .textgen import (  # noqa: F401
    CONFIGS,
    config_text,
    batch_docs,
    latency_sample,
    training_text,
    stress_text,
)
