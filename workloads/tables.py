"""Load the stored merge tables of the benchmark configurations.

The files are written by the oracle's trainer (``oracle/train_tables.py``);
this module only reads them.  Configuration 5 uses the table of configuration 4.
"""

import os

import numpy as np

from .textgen import CONFIGS

TABLE_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tables")


def table_path(k: int) -> str:
    k = CONFIGS[k].get("table_from", k)
    return os.path.join(TABLE_DIR, "c%d.npz" % k)


def load_table(k: int):
    """(merges int32 [M,3], vocab_bytes uint8 [*], vocab_offsets int64 [V+1]) of configuration ``k``."""
    with np.load(table_path(k), allow_pickle=False) as z:
        return z["merges"].copy(), z["vocab_bytes"].copy(), z["vocab_offsets"].copy()


def vocab_list(vocab_bytes, vocab_offsets) -> list:
    """The vocabulary as a list of ``bytes`` (index = ID)."""
    vb = bytes(vocab_bytes)
    off = [int(x) for x in vocab_offsets]
    return [vb[off[i]:off[i + 1]] for i in range(len(off) - 1)]
