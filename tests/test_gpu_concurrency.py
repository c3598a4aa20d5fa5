"""Several streams and host threads on one handle.

A handle keeps one workspace per stream, so requests on different streams may
be in flight at the same time, from one host thread or from several.  Each
stream's requests are enqueued without synchronising the others, on two
handles (two tables and patterns) at once; every output is compared with the
oracle.  Tiles wait only on tiles that took a lower ticket of their own
launch, so launches that share the chip make progress.
"""

import threading

import numpy as np
import pytest

from conftest import config_bytes, oracle_ids, oracle_table, pattern_of

pytestmark = pytest.mark.gpu


def _slices(k, n, size):
    """n distinct slices of configuration k's text, cut at character boundaries."""
    text = config_bytes(k).decode("utf-8")
    step = (len(text) - size) // max(1, n - 1)
    return [text[i * step:i * step + size].encode("utf-8") for i in range(n)]


_WANT = {}


def _want(k, data):
    key = (k, data)
    if key not in _WANT:
        _WANT[key] = oracle_ids(data, oracle_table(k), pattern_of(k))
    return _WANT[key]


def test_streams_in_flight_together(gpu):
    torch = gpu
    from conftest import lib_tokenizer

    jobs = []  # (stream, k, data)
    streams = [torch.cuda.Stream() for _ in range(6)]
    for j, s in enumerate(streams):
        k = 3 if j % 2 == 0 else 4
        for data in _slices(k, 3, 150_000 + 20_000 * j):
            jobs.append((s, k, data))
    bufs = []
    for s, k, data in jobs:
        with torch.cuda.stream(s):
            d_in = torch.from_numpy(np.frombuffer(data, dtype=np.uint8).copy()).to("cuda", non_blocking=False)
            d_out = torch.empty(len(data), dtype=torch.int32, device="cuda")
            d_len = torch.zeros(1, dtype=torch.int64, device="cuda")
        bufs.append((d_in, d_out, d_len))
    torch.cuda.synchronize()
    # enqueue everything, round-robin over the streams, then wait once
    for (s, k, data), (d_in, d_out, d_len) in zip(jobs, bufs):
        lib_tokenizer(k).encode_device(d_in, len(data), d_out, d_len, s.cuda_stream)
    torch.cuda.synchronize()
    for (s, k, data), (d_in, d_out, d_len) in zip(jobs, bufs):
        T = int(d_len.item())
        assert d_out[:T].cpu().numpy().tolist() == _want(k, data), (k, len(data))


def test_host_threads_with_own_streams(gpu):
    torch = gpu
    from conftest import lib_tokenizer

    work = {}
    for t in range(4):
        k = 3 if t % 2 == 0 else 4
        work[t] = (k, _slices(k, 4, 60_000 + 7_000 * t))
    for k, datas in work.values():  # oracle and handles first, outside the threads
        lib_tokenizer(k)
        for d in datas:
            _want(k, d)
    results, errors = {}, []

    def run(t):
        try:
            k, datas = work[t]
            s = torch.cuda.Stream()
            tok = lib_tokenizer(k)
            out = []
            for _ in range(3):
                for d in datas:
                    out.append(tok.encode(d, s.cuda_stream).tolist())
            results[t] = out
        except Exception as e:  # reported in the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=run, args=(t,)) for t in work]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    for t, (k, datas) in work.items():
        got = results[t]
        assert len(got) == 3 * len(datas)
        for i, g in enumerate(got):
            assert g == _want(k, datas[i % len(datas)]), (t, i)
