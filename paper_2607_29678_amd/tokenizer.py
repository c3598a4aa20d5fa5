"""Python binding of the C ABI: argument marshalling only.

Every step of tokenization runs in the HIP library; these wrappers convert
Python/numpy arguments to pointers and sizes and raise on error status.
Device-memory entry points take raw device addresses (ints) or objects with a
``data_ptr()`` method (e.g. torch tensors), and a HIP stream handle as an int
(e.g. ``torch.cuda.current_stream().cuda_stream``) or None for the null stream.
"""

import ctypes

import numpy as np

from . import _lib

GPT2 = _lib.TT_PATTERN_GPT2
CL100K = _lib.TT_PATTERN_CL100K
PATTERNS = {"gpt2": GPT2, "cl100k": CL100K}


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return ctypes.c_void_p(x)
    if hasattr(x, "data_ptr"):
        return ctypes.c_void_p(x.data_ptr())
    if isinstance(x, np.ndarray):
        return x.ctypes.data_as(ctypes.c_void_p)
    raise TypeError("cannot take the address of %r" % type(x))


def _stream(s):
    return None if s is None else ctypes.c_void_p(int(s))


def _u8(data):
    if isinstance(data, np.ndarray):
        return np.ascontiguousarray(data, dtype=np.uint8)
    return np.frombuffer(bytes(data), dtype=np.uint8)


class Tokenizer:
    """An immutable tokenizer handle (``tt_create`` / ``tt_destroy``)."""

    def __init__(self, merges, vocab_bytes, vocab_offsets, pattern="gpt2"):
        lib = _lib.load()
        self._lib = lib
        pat = PATTERNS[pattern] if isinstance(pattern, str) else int(pattern)
        m = np.ascontiguousarray(np.asarray(merges, dtype=np.int32).reshape(-1, 3))
        vb = np.ascontiguousarray(np.asarray(vocab_bytes, dtype=np.uint8))
        vo = np.ascontiguousarray(np.asarray(vocab_offsets, dtype=np.int64))
        h = ctypes.c_void_p()
        st = lib.tt_create(_ptr(m), len(m), _ptr(vb) if vb.size else None, _ptr(vo), len(vo) - 1, pat,
                           ctypes.byref(h))
        _lib.check(st, "tt_create")
        self._h = h
        self.pattern = pat
        self.n_merges = len(m)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.tt_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # -- host entry points -------------------------------------------------
    def encode(self, data, stream=None) -> np.ndarray:
        """``tt_encode``: token IDs (int32) of one UTF-8 request."""
        src = _u8(data)
        out = np.empty(max(1, src.size), dtype=np.int32)
        n = ctypes.c_int64(0)
        st = self._lib.tt_encode(self._h, _ptr(src) if src.size else None, src.size, _ptr(out), ctypes.byref(n),
                                 _stream(stream))
        _lib.check(st, "tt_encode")
        return out[: n.value].copy()

    def encode_spans(self, data, stream=None):
        """``tt_encode_spans``: (IDs int32 [T], spans int32 [T, 4]) of one UTF-8 request; a span is
        (byte begin, byte end, char begin, char end)."""
        src = _u8(data)
        ids = np.empty(max(1, src.size), dtype=np.int32)
        spans = np.empty((max(1, src.size), 4), dtype=np.int32)
        n = ctypes.c_int64(0)
        st = self._lib.tt_encode_spans(self._h, _ptr(src) if src.size else None, src.size, _ptr(ids), _ptr(spans),
                                       ctypes.byref(n), _stream(stream))
        _lib.check(st, "tt_encode_spans")
        return ids[: n.value].copy(), spans[: n.value].copy()

    def encode_batch(self, docs, stream=None):
        """``tt_encode_batch``: list of int32 ID arrays, one per document."""
        parts = [bytes(d) for d in docs]
        offs = np.zeros(len(parts) + 1, dtype=np.int64)
        np.cumsum([len(p) for p in parts], out=offs[1:])
        src = np.frombuffer(b"".join(parts), dtype=np.uint8)
        out = np.empty(max(1, src.size), dtype=np.int32)
        out_off = np.zeros(len(parts) + 1, dtype=np.int64)
        st = self._lib.tt_encode_batch(self._h, _ptr(src) if src.size else None, _ptr(offs), len(parts),
                                       _ptr(out), _ptr(out_off), _stream(stream))
        _lib.check(st, "tt_encode_batch")
        return [out[out_off[j]:out_off[j + 1]].copy() for j in range(len(parts))]

    def pretokenize(self, data, stream=None) -> np.ndarray:
        """``tt_pretokenize``: UTF-8 byte offset of the first byte of every piece (int64)."""
        src = _u8(data)
        out = np.empty(max(1, src.size), dtype=np.int64)
        n = ctypes.c_int64(0)
        st = self._lib.tt_pretokenize(self._h, _ptr(src) if src.size else None, src.size, _ptr(out),
                                      ctypes.byref(n), _stream(stream))
        _lib.check(st, "tt_pretokenize")
        return out[: n.value].copy()

    # -- device entry point ------------------------------------------------
    def encode_device(self, d_utf8, length, d_out_ids, d_out_len, stream=None):
        """``tt_encode_device``: enqueue on ``stream``; d_out_len (int64) receives T or -error."""
        st = self._lib.tt_encode_device(self._h, _ptr(d_utf8), int(length), _ptr(d_out_ids), _ptr(d_out_len),
                                        _stream(stream))
        _lib.check(st, "tt_encode_device")

    def encode_spans_device(self, d_utf8, length, d_out_ids, d_out_spans, d_out_len, stream=None):
        """``tt_encode_spans_device``: enqueue on ``stream``; d_out_spans holds 4 int32 per token."""
        st = self._lib.tt_encode_spans_device(self._h, _ptr(d_utf8), int(length), _ptr(d_out_ids),
                                              _ptr(d_out_spans), _ptr(d_out_len), _stream(stream))
        _lib.check(st, "tt_encode_spans_device")


    # -- measurement -------------------------------------------------------
    def set_profiling(self, n_calls=1):
        """``tt_set_profiling``: keep the stage events of the last ``n_calls`` calls (0 = off)."""
        _lib.check(self._lib.tt_set_profiling(self._h, int(n_calls)), "tt_set_profiling")

    def stage_times(self, stream=None, max_calls=4096) -> list:
        """``tt_stage_times``: one {stage name: ms} dict per recorded call on ``stream``, oldest first."""
        ns = len(_lib.STAGES)
        out = np.zeros(ns * max_calls, dtype=np.float64)
        n = ctypes.c_int32(0)
        _lib.check(self._lib.tt_stage_times(self._h, _stream(stream), _ptr(out), out.size, ctypes.byref(n)),
                   "tt_stage_times")
        return [{_lib.STAGES[i]: float(out[c * ns + i]) for i in range(ns)} for c in range(n.value // ns)]


def status_string(status: int) -> str:
    return _lib.load().tt_status_string(status).decode()
