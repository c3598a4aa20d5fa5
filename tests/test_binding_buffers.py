"""The binding's reusable output buffers (``tokenizer._ResultBuffers``), on the CPU.

``Tokenizer.encode`` hands out views of these buffers; a buffer may be handed
out again only when no array refers to it.  Checked here without a GPU: a kept
result or any view of it keeps its buffer out of use, a free buffer is reused,
a larger request replaces the smallest free buffer when the pool is full, and
threads never receive the same buffer at once.
"""

import threading

import numpy as np

from paper_2607_29678_amd.tokenizer import _ResultBuffers


def test_views_keep_their_buffer():
    p = _ResultBuffers()
    a, kept = p.take(100)
    assert kept and a.size >= 100
    r = a[:40]
    rr = r[5:][::2]  # a view of a view
    del a, r
    b, _ = p.take(100)
    assert not np.shares_memory(b, rr)
    del b
    c, _ = p.take(100)  # the second buffer is free again
    assert not np.shares_memory(c, rr)
    del rr, c
    d, _ = p.take(10)   # both free now: the first one is reused
    assert d is p._bufs[0]


def test_full_pool_and_replacement():
    p = _ResultBuffers()
    held = [p.take(100)[0][:50] for _ in range(p.KEEP)]
    b, kept = p.take(100)
    assert not kept  # every kept buffer is in use: a buffer of its own
    del b
    del held[0]
    big, kept = p.take(1000)
    assert kept and big.size >= 1000  # took the place of the free small buffer
    assert sorted(x.size for x in p._bufs)[-1] == big.size
    assert all(not np.shares_memory(big, h) for h in held)


def test_large_results_are_not_kept():
    p = _ResultBuffers()
    b, kept = p.take(p.MAX_ENTRIES + 1)
    assert not kept and b.size == p.MAX_ENTRIES + 1
    assert p._bufs == []


def test_threads_never_share_a_buffer():
    p = _ResultBuffers()
    errors = []

    def run(tag):
        for i in range(3000):
            b, _ = p.take(64 + (i % 7))
            b[:64] = tag
            if not (b[:64] == tag).all():
                errors.append(tag)
            if i % 5 == 0:
                keep = b[:8]  # sometimes keep a view for a while
                b = None
                keep[:] = tag
                if not (keep == tag).all():
                    errors.append(tag)

    th = [threading.Thread(target=run, args=(t + 1,)) for t in range(6)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors
