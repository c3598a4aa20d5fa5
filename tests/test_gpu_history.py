"""History independence and the comparator itself.

A call's output must not depend on what the handle or its stream's workspace
did before: the workspace keeps epoch-tagged words, a grown capacity and
pinned staging that holds the previous request's bytes and IDs.  Requests of
different sizes and IDs-per-byte ratios go through one handle and one stream
in turn, through the host entry point with pageable and pinned caller
buffers and through the device entry point; each result is compared with the
oracle and with a fresh handle's.

The comparator of the parity tests is checked too: a mutated ID or a moved
piece boundary in a real GPU result must be reported, at its position.
"""

import random

import numpy as np
import pytest

from conftest import config_bytes, lib_tokenizer, oracle_ids, oracle_table, stored_table

pytestmark = pytest.mark.gpu


def _first_diff(a, b):
    n = min(len(a), len(b))
    for i in range(n):
        if a[i] != b[i]:
            return i
    return n if len(a) != len(b) else -1


def _cjk(n, seed):
    rng = random.Random(seed)
    return "".join(chr(rng.randint(0x4E00, 0x9FA5)) for _ in range(n)).encode("utf-8")


def test_history_independence(gpu):
    from paper_2607_29678_amd import Tokenizer

    torch = gpu
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream(0)
    sid = stream.cuda_stream
    m, vb, vo = stored_table(3)
    x = config_bytes(3)                 # 1,000,000 bytes, about 0.31 IDs per byte
    y = config_bytes(1)                 # 10,000 bytes
    z = _cjk(30_000, 7)                 # 90,000 bytes, about one ID per byte under this table
    table = oracle_table(3)
    want = {name: oracle_ids(d, table, "gpt2") for name, d in (("x", x), ("y", y), ("z", z))}
    data = {"x": x, "y": y, "z": z}
    order = ["x", "y", "x", "z", "x", "y", "z", "z", "x"]
    with Tokenizer(m, vb, vo, "gpt2") as tok:
        cap = len(x)
        out = np.full(cap, -3, dtype=np.int32)
        pin_out = torch.full((cap,), -3, dtype=torch.int32).pin_memory()
        d_out = torch.full((cap,), -3, dtype=torch.int32, device="cuda:0")
        d_len = torch.zeros(1, dtype=torch.int64, device="cuda:0")
        for step, name in enumerate(order):
            d = data[name]
            n = tok.encode_into(d, out, sid)
            assert out[:n].tolist() == want[name], "pageable, step %d (%s)" % (step, name)
            pin_in = torch.from_numpy(np.frombuffer(d, dtype=np.uint8).copy()).pin_memory()
            n = tok.encode_into(pin_in, pin_out, sid)
            assert pin_out[:n].tolist() == want[name], "pinned, step %d (%s)" % (step, name)
            d_in = torch.from_numpy(np.frombuffer(d, dtype=np.uint8).copy()).to("cuda:0")
            tok.encode_device(d_in, len(d), d_out, d_len, sid)
            stream.synchronize()
            n = int(d_len.item())
            assert d_out[:n].cpu().tolist() == want[name], "device, step %d (%s)" % (step, name)
    # a fresh handle on another stream gives the same
    s2 = torch.cuda.Stream()
    with Tokenizer(m, vb, vo, "gpt2") as fresh:
        for name in ("z", "x"):
            assert fresh.encode(data[name], s2.cuda_stream).tolist() == want[name]


def test_comparator_flags_a_mutated_id(gpu):
    k = 1
    got = lib_tokenizer(k).encode(config_bytes(k)).tolist()
    want = oracle_ids(config_bytes(k), oracle_table(k), "gpt2")
    assert _first_diff(got, want) == -1
    rng = random.Random(5)
    for _ in range(20):
        i = rng.randrange(len(got))
        bad = list(got)
        bad[i] = bad[i] + 1
        assert _first_diff(bad, want) == i
        assert _first_diff(got[:i] + got[i + 1:], want) == i  # a dropped ID


def test_comparator_flags_a_moved_boundary(gpu):
    from oracle.pretok import piece_byte_starts

    k = 1
    data = config_bytes(k)
    got = lib_tokenizer(k).pretokenize(data).tolist()
    want = piece_byte_starts(data.decode("utf-8"), "gpt2")
    assert _first_diff(got, want) == -1
    rng = random.Random(6)
    for _ in range(20):
        i = rng.randrange(1, len(got) - 1)
        moved = list(got)
        moved[i] += 1  # the boundary one byte later (still between its neighbours or equal to the next)
        assert _first_diff(moved, want) == i
        merged = got[:i] + got[i + 1:]  # two pieces joined
        assert _first_diff(merged, want) == i
