"""Results of the binding's ``Tokenizer.encode`` stay valid while they are kept.

``encode`` returns views of output buffers that later calls reuse once no
array refers to them.  Here results are kept across many later calls (more
than the buffers kept), views of views outlive their parents, and two host
threads encode at once on their own streams; every result is compared with
the oracle after all calls.
"""

import threading

import numpy as np
import pytest

from conftest import config_bytes, lib_tokenizer, oracle_ids, oracle_table

pytestmark = pytest.mark.gpu

K = 3


def _texts(n, seed):
    text = config_bytes(K).decode("utf-8")
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        size = int(rng.choice([1, 17, 3000, 40_000, 120_000]))
        a = int(rng.integers(0, len(text) - size))
        out.append(text[a:a + size].encode("utf-8"))
    return out


def _want(data):
    return np.asarray(oracle_ids(data, oracle_table(K), "gpt2"), dtype=np.int64)


def test_results_kept_across_later_calls(gpu):
    tok = lib_tokenizer(K)
    texts = _texts(10, 1)
    kept = [tok.encode(t) for t in texts]           # ten results alive at once
    parts = [r[: len(r) // 2][1:] for r in kept[:3]]  # views of views of the first three
    del kept[:3]
    for t in _texts(12, 2):                          # later calls, results dropped at once
        tok.encode(t)
    for r, t in zip(kept, texts[3:]):
        assert np.array_equal(np.asarray(r, dtype=np.int64), _want(t))
    for p, t in zip(parts, texts[:3]):
        w = _want(t)
        assert np.array_equal(np.asarray(p, dtype=np.int64), w[: len(w) // 2][1:])


def test_results_of_two_threads(gpu):
    torch = gpu
    tok = lib_tokenizer(K)
    jobs = [_texts(6, 10 + j) for j in range(2)]
    results = [[], []]
    errors = []

    def run(j):
        try:
            s = torch.cuda.Stream()
            for t in jobs[j]:
                results[j].append(tok.encode(t, s.cuda_stream))
        except Exception as e:  # reported below
            errors.append(e)

    th = [threading.Thread(target=run, args=(j,)) for j in range(2)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    assert not errors, errors
    for j in range(2):
        for r, t in zip(results[j], jobs[j]):
            assert np.array_equal(np.asarray(r, dtype=np.int64), _want(t))
