"""Python binding of the C ABI: argument marshalling only.

Every step of tokenization runs in the HIP library; these wrappers convert
Python/numpy arguments to pointers and sizes and raise on error status.
Device-memory entry points take raw device addresses (ints) or objects with a
``data_ptr()`` method (e.g. torch tensors), and a HIP stream handle as an int
(e.g. ``torch.cuda.current_stream().cuda_stream``) or None for the null stream.
"""

import ctypes
import sys
import threading

import numpy as np

from . import _lib

GPT2 = _lib.TT_PATTERN_GPT2
CL100K = _lib.TT_PATTERN_CL100K
O200K = _lib.TT_PATTERN_O200K
DEEPSEEK = _lib.TT_PATTERN_DEEPSEEK
PATTERNS = {"gpt2": GPT2, "cl100k": CL100K, "o200k": O200K, "deepseek": DEEPSEEK}


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return ctypes.c_void_p(x)
    if hasattr(x, "data_ptr"):
        return ctypes.c_void_p(x.data_ptr())
    if isinstance(x, np.ndarray):
        # (the buffer protocol is the cheapest route for a writable array; numpy's
        # ctypes attribute costs a few microseconds per call)
        if x.flags.writeable and x.flags.c_contiguous and x.nbytes:
            return ctypes.c_void_p(ctypes.addressof(ctypes.c_ubyte.from_buffer(x)))
        return ctypes.c_void_p(x.ctypes.data)
    raise TypeError("cannot take the address of %r" % type(x))


def _stream(s):
    return None if s is None else ctypes.c_void_p(int(s))


def _shrunk(a, n):
    """``a`` (a fresh array this module owns) cut to its first n rows in place:
    the allocation shrinks without a copy of the rows kept."""
    a.resize((n,) + a.shape[1:], refcheck=False)
    return a


class _ResultBuffers:
    """Output arrays of ``Tokenizer.encode``, reused once nothing refers to them.

    A fresh array's pages are mapped on first touch, while the library copies
    the IDs into it, and those faults cost more than the copy.  ``encode``
    returns a view of a buffer kept here; a later call takes the buffer again
    only when no array refers to it any more (every view of it holds a
    reference), so a result stays valid for as long as the caller keeps it.
    """

    KEEP = 4                # buffers kept
    MAX_ENTRIES = 1 << 24   # larger results get an array of their own

    def __init__(self):
        self._bufs = []
        self._lock = threading.Lock()

    def take(self, n):
        """An int32 array of at least n entries that nothing else refers to,
        and whether it is one of the kept buffers."""
        if n > self.MAX_ENTRIES:
            return np.empty(n, dtype=np.int32), False
        with self._lock:
            free = []
            for i in range(len(self._bufs)):
                b = self._bufs[i]
                # references: the list, b and the call's argument
                if sys.getrefcount(b) == 3:
                    if b.size >= n:
                        return b, True
                    free.append(i)
            # a new buffer, with room for requests a little longer than this one,
            # kept in place of the smallest free one when the pool is full
            b = np.empty(min(n + n // 4, max(n, self.MAX_ENTRIES)), dtype=np.int32)
            if len(self._bufs) < self.KEEP:
                self._bufs.append(b)
                return b, True
            if free:
                self._bufs[min(free, key=lambda i: self._bufs[i].size)] = b
                return b, True
            return b, False


def _u8(data):
    if isinstance(data, np.ndarray):
        return np.ascontiguousarray(data, dtype=np.uint8)
    return np.frombuffer(bytes(data), dtype=np.uint8)


class Tokenizer:
    """An immutable tokenizer handle (``tt_create`` / ``tt_destroy``)."""

    def __init__(self, merges, vocab_bytes, vocab_offsets, pattern="gpt2", ignore_merges=False, added=None):
        """``added``: optional list of (literal bytes or str, ID) added tokens (``tt_create_ex``)."""
        lib = _lib.load()
        self._lib = lib
        pat = PATTERNS[pattern] if isinstance(pattern, str) else int(pattern)
        m = np.ascontiguousarray(np.asarray(merges, dtype=np.int32).reshape(-1, 3))
        vb = np.ascontiguousarray(np.asarray(vocab_bytes, dtype=np.uint8))
        vo = np.ascontiguousarray(np.asarray(vocab_offsets, dtype=np.int64))
        h = ctypes.c_void_p()
        if ignore_merges or added:
            lits = [(x.encode("utf-8") if isinstance(x, str) else bytes(x), int(i)) for x, i in (added or [])]
            ab = np.frombuffer(b"".join(x for x, _ in lits) or b"\0", dtype=np.uint8).copy()
            ao = np.zeros(len(lits) + 1, dtype=np.int64)
            np.cumsum([len(x) for x, _ in lits], out=ao[1:])
            ai = np.asarray([i for _, i in lits] or [0], dtype=np.int32)
            self._added = (ab, ao, ai)  # kept alive for the call
            opt = _lib.Options(int(bool(ignore_merges)), len(lits), _ptr(ab).value, _ptr(ao).value, _ptr(ai).value)
            st = lib.tt_create_ex(_ptr(m), len(m), _ptr(vb) if vb.size else None, _ptr(vo), len(vo) - 1, pat,
                                  ctypes.byref(opt), ctypes.byref(h))
        else:
            st = lib.tt_create(_ptr(m), len(m), _ptr(vb) if vb.size else None, _ptr(vo), len(vo) - 1, pat,
                               ctypes.byref(h))
        _lib.check(st, "tt_create")
        self._h = h
        self.pattern = pat
        self.n_merges = len(m)
        self.vocab_size = len(vo) - 1  # caller IDs lie in [0, vocab_size)
        self._results = _ResultBuffers()

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
        """``tt_encode``: token IDs (int32) of one UTF-8 request.  The result may
        be a view of a larger buffer that a later call reuses once no array
        refers to it."""
        src = _u8(data)
        out, kept = self._results.take(max(1, src.size))
        n = ctypes.c_int64(0)
        st = self._lib.tt_encode(self._h, _ptr(src) if src.size else None, src.size, _ptr(out), ctypes.byref(n),
                                 _stream(stream))
        _lib.check(st, "tt_encode")
        return out[: n.value] if kept else _shrunk(out, n.value)

    def encode_into(self, data, out, stream=None) -> int:
        """``tt_encode`` into a caller-provided int32 array ``out`` (numpy or a CPU torch tensor, at
        least ``max(1, len(data))`` entries, reusable across calls; pinned memory is copied into
        directly).  Returns the number of IDs written."""
        if hasattr(data, "data_ptr"):  # a CPU torch tensor of bytes (pinned or not)
            if repr(data.dtype) != "torch.uint8" or not data.is_contiguous() or data.is_cuda:
                raise ValueError("data must be a contiguous uint8 CPU tensor")
            src, size = data, data.numel()
        else:
            src = _u8(data)
            size = src.size
        if hasattr(out, "data_ptr"):
            ok = repr(out.dtype) == "torch.int32" and out.is_contiguous() and not out.is_cuda and out.numel() >= max(1, size)
        else:
            ok = out.dtype == np.int32 and out.flags["C_CONTIGUOUS"] and out.size >= max(1, size)
        if not ok:
            raise ValueError("out must be a contiguous int32 host array of at least max(1, len(data)) entries")
        n = ctypes.c_int64(0)
        st = self._lib.tt_encode(self._h, _ptr(src) if size else None, size, _ptr(out), ctypes.byref(n),
                                 _stream(stream))
        _lib.check(st, "tt_encode")
        return n.value

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
        return _shrunk(ids, n.value), _shrunk(spans, n.value)

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
        return _shrunk(out, n.value)

    # -- device entry point ------------------------------------------------
    def encode_device(self, d_utf8, length, d_out_ids, d_out_len, stream=None):
        """``tt_encode_device``: enqueue on ``stream``; d_out_len (int64) receives T or -error."""
        st = self._lib.tt_encode_device(self._h, _ptr(d_utf8), int(length), _ptr(d_out_ids), _ptr(d_out_len),
                                        _stream(stream))
        _lib.check(st, "tt_encode_device")

    def encode_device_noalloc(self, d_utf8, length, d_out_ids, d_out_len, stream=None):
        """``tt_encode_device_noalloc``: as ``encode_device``, with the library's fixed per-GPU
        workspace (no allocation; at most ``TT_NOALLOC_MAX_BYTES`` bytes; overlapping calls on one GPU
        race)."""
        st = self._lib.tt_encode_device_noalloc(self._h, _ptr(d_utf8), int(length), _ptr(d_out_ids),
                                                _ptr(d_out_len), _stream(stream))
        _lib.check(st, "tt_encode_device_noalloc")

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


class Session:
    """Incremental repair over a growing request (``tt_session_*``).

    After every ``append`` the session's IDs equal full tokenization of the
    whole text; ``append`` returns the ``tt_append_info`` fields as a dict.
    """

    def __init__(self, tokenizer: Tokenizer, window_chars: int = 0):
        self._lib = tokenizer._lib
        self._tok = tokenizer  # the handle must outlive the session
        h = ctypes.c_void_p()
        _lib.check(self._lib.tt_session_create(tokenizer._h, int(window_chars), ctypes.byref(h)),
                   "tt_session_create")
        self._s = h

    def close(self):
        if getattr(self, "_s", None):
            self._lib.tt_session_destroy(self._s)
            self._s = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def append(self, data, stream=None) -> dict:
        src = _u8(data)
        info = _lib.AppendInfo()
        st = self._lib.tt_session_append(self._s, _ptr(src) if src.size else None, src.size, ctypes.byref(info),
                                         _stream(stream))
        _lib.check(st, "tt_session_append")
        return {k: int(getattr(info, k)) for k, _ in _lib.AppendInfo._fields_}

    def info(self) -> dict:
        b, c, t = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int64(0)
        _lib.check(self._lib.tt_session_info(self._s, ctypes.byref(b), ctypes.byref(c), ctypes.byref(t)),
                   "tt_session_info")
        return {"bytes": b.value, "chars": c.value, "tokens": t.value}

    def tokens(self, start=0, count=None):
        """(IDs int32 [count], spans int32 [count, 4]) of tokens [start, start + count)."""
        n = self.info()["tokens"]
        count = n - start if count is None else count
        ids = np.empty(max(1, count), dtype=np.int32)
        spans = np.empty((max(1, count), 4), dtype=np.int32)
        _lib.check(self._lib.tt_session_tokens(self._s, int(start), int(count), _ptr(ids), _ptr(spans)),
                   "tt_session_tokens")
        return _shrunk(ids, count), _shrunk(spans, count)

    def ids(self) -> np.ndarray:
        return self.tokens()[0]


def sync_boundaries(data, pattern="gpt2") -> np.ndarray:
    """``tt_sync_boundaries``: uint8 mask of the synchronizing byte positions of a text (host only)."""
    lib = _lib.load()
    pat = PATTERNS[pattern] if isinstance(pattern, str) else int(pattern)
    src = _u8(data)
    out = np.zeros(max(1, src.size), dtype=np.uint8)
    _lib.check(lib.tt_sync_boundaries(pat, _ptr(src) if src.size else None, src.size, _ptr(out)),
               "tt_sync_boundaries")
    return _shrunk(out, src.size)


def splice_plan(text, a_len, x, c_ids, c_spans, f_ids, f_spans, max_token_chars, pattern="gpt2"):
    """``tt_splice_plan``: (keep_c, from_f) when the window is admitted, else None (host only)."""
    lib = _lib.load()
    pat = PATTERNS[pattern] if isinstance(pattern, str) else int(pattern)
    src = _u8(text)
    ci = np.ascontiguousarray(c_ids, dtype=np.int32)
    cs = np.ascontiguousarray(np.asarray(c_spans, dtype=np.int32).reshape(-1, 4))
    fi = np.ascontiguousarray(f_ids, dtype=np.int32)
    fs = np.ascontiguousarray(np.asarray(f_spans, dtype=np.int32).reshape(-1, 4))
    kc, ff = ctypes.c_int64(0), ctypes.c_int64(0)
    st = lib.tt_splice_plan(pat, _ptr(src), src.size, int(a_len), int(x), _ptr(ci), _ptr(cs), len(ci), _ptr(fi),
                            _ptr(fs), len(fi), int(max_token_chars), ctypes.byref(kc), ctypes.byref(ff))
    if st < 0:
        _lib.check(st, "tt_splice_plan")
    return (kc.value, ff.value) if st == 1 else None


def status_string(status: int) -> str:
    return _lib.load().tt_status_string(status).decode()
