"""The C ABI without a GPU: the library loads, exports what the header declares,
and rejects invalid handles and tables before touching the device."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_29678_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "toktier.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tt_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    assert _declared() == sorted(["tt_create", "tt_create_ex", "tt_destroy", "tt_encode", "tt_encode_device",
                                  "tt_encode_device_noalloc", "tt_encode_batch",
                                  "tt_encode_spans", "tt_encode_spans_device", "tt_pretokenize",
                                  "tt_status_string", "tt_info", "tt_set_profiling", "tt_stage_times",
                                  "tt_session_create", "tt_session_destroy", "tt_session_append",
                                  "tt_session_tokens", "tt_session_info", "tt_sync_boundaries", "tt_splice_plan"])


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_lib.SIGNATURES) == set(_declared())


def test_product_library_has_no_phase_stamps():
    # the per-phase clock stamps exist only in the diagnostic build
    # (phase_timeline.py, TT_PHASE_STAMPS); the product library exports none
    lib = _lib.load()
    assert not hasattr(lib, "tt_phase_stamps")


def test_status_strings():
    lib = _lib.load()
    for code in _lib.STATUS:
        assert lib.tt_status_string(code)
    assert lib.tt_status_string(-5).decode() == "input is not valid UTF-8"


def _base_vocab():
    vb = np.arange(256, dtype=np.uint8)
    vo = np.arange(257, dtype=np.int64)
    return vb, vo


def _create(merges, vb, vo, pattern=0):
    lib = _lib.load()
    m = np.ascontiguousarray(np.asarray(merges, dtype=np.int32).reshape(-1, 3))
    h = ctypes.c_void_p()
    st = lib.tt_create(m.ctypes.data_as(ctypes.c_void_p) if len(m) else None, len(m),
                       vb.ctypes.data_as(ctypes.c_void_p), vo.ctypes.data_as(ctypes.c_void_p), len(vo) - 1,
                       pattern, ctypes.byref(h))
    return st, h


def _vocab_with(extra):
    toks = [bytes([i]) for i in range(256)] + extra
    vb = np.frombuffer(b"".join(toks), dtype=np.uint8).copy()
    vo = np.zeros(len(toks) + 1, dtype=np.int64)
    np.cumsum([len(t) for t in toks], out=vo[1:])
    return vb, vo


def test_create_rejects_bad_pattern():
    vb, vo = _base_vocab()
    assert _create([], vb, vo, pattern=7)[0] == -2


def test_create_rejects_out_of_range():
    vb, vo = _vocab_with([b"ab"])
    assert _create([(97, 98, 300)], vb, vo)[0] == -3
    assert _create([(-1, 98, 256)], vb, vo)[0] == -3


def test_create_rejects_duplicate_pair():
    vb, vo = _vocab_with([b"ab", b"ab"])
    assert _create([(97, 98, 256), (97, 98, 257)], vb, vo)[0] == -3


def test_create_rejects_non_proper_operand():
    vb, vo = _vocab_with([b"abc", b"ab"])
    # merge 0 uses 257 ("ab") before any merge produced it
    assert _create([(257, 99, 256), (97, 98, 257)], vb, vo)[0] == -3


def test_create_rejects_repeated_result():
    vb, vo = _vocab_with([b"ab", b"abc", b"bc"])
    assert _create([(97, 98, 256), (98, 99, 258), (97, 258, 256)], vb, vo)[0] == -3


def test_create_rejects_vocab_mismatch():
    vb, vo = _vocab_with([b"ba"])
    assert _create([(97, 98, 256)], vb, vo)[0] == -4


def test_create_rejects_missing_byte():
    toks = [bytes([i]) for i in range(255)] + [b"xy"]
    vb = np.frombuffer(b"".join(toks), dtype=np.uint8).copy()
    vo = np.zeros(len(toks) + 1, dtype=np.int64)
    np.cumsum([len(t) for t in toks], out=vo[1:])
    assert _create([], vb, vo)[0] == -4


def test_null_arguments():
    lib = _lib.load()
    n = ctypes.c_int64(0)
    assert lib.tt_encode(None, None, 0, None, ctypes.byref(n), None) == -1
    assert lib.tt_pretokenize(None, None, 0, None, ctypes.byref(n), None) == -1
    assert lib.tt_encode_device(None, None, 0, None, None, None) == -1
    assert lib.tt_encode_batch(None, None, None, 0, None, None, None) == -1
    assert lib.tt_create(None, 0, None, None, 256, 0, None) == -1
    lib.tt_destroy(None)


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", "/nonexistent/libtoktier.so")
    with pytest.raises(ImportError):
        _lib.load()


def _create_ex(lits, ids, ignore=0):
    lib = _lib.load()
    vb, vo = _base_vocab()
    ab = np.frombuffer(b"".join(lits) or b"\0", dtype=np.uint8).copy()
    ao = np.zeros(len(lits) + 1, dtype=np.int64)
    np.cumsum([len(x) for x in lits], out=ao[1:])
    ai = np.asarray(ids or [0], dtype=np.int32)
    opt = _lib.Options(ignore, len(lits), ab.ctypes.data, ao.ctypes.data, ai.ctypes.data)
    h = ctypes.c_void_p()
    return lib.tt_create_ex(None, 0, vb.ctypes.data_as(ctypes.c_void_p), vo.ctypes.data_as(ctypes.c_void_p),
                            len(vo) - 1, 0, ctypes.byref(opt), ctypes.byref(h))


def test_create_ex_rejects_bad_literals():
    """Literals are validated on the host before any device work."""
    assert _create_ex([b"<a>", b"<a>"], [1, 2]) == -9      # duplicate
    assert _create_ex([b"<a>", b""], [1, 2]) == -9         # empty
    assert _create_ex([b"<\xff>"], [1]) == -9              # not UTF-8
    assert _create_ex([b"\xe2\x82"], [1]) == -9            # truncated character
    assert _create_ex([b"<a>"], [-1]) == -9                # negative ID
    assert _create_ex([b"x" * 1025], [1]) == -9            # longer than TT_MAX_ADDED_BYTES


def test_host_only_exports_need_no_gpu():
    from paper_2607_29678_amd import sync_boundaries

    assert list(sync_boundaries(b"ab 1", "gpt2")) == [0, 0, 1, 0]
