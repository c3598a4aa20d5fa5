"""ctypes declarations of the C ABI in ``include/toktier.h``.

Loading fails loudly when ``libtoktier.so`` has not been built: there is no
fallback implementation in this package.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtoktier.so")

TT_OK = 0
TT_PATTERN_GPT2 = 0
TT_PATTERN_CL100K = 1
TT_PATTERN_O200K = 2
TT_PATTERN_DEEPSEEK = 3
TT_MAX_BYTES = 1 << 30
TT_NOALLOC_MAX_BYTES = 1 << 21

STATUS = {
    0: "TT_OK",
    -1: "TT_ERR_NULL_ARG",
    -2: "TT_ERR_BAD_PATTERN",
    -3: "TT_ERR_BAD_MERGES",
    -4: "TT_ERR_BAD_VOCAB",
    -5: "TT_ERR_INVALID_UTF8",
    -6: "TT_ERR_TOO_LARGE",
    -7: "TT_ERR_HIP",
    -8: "TT_ERR_OOM",
    -9: "TT_ERR_BAD_ARG",
}

# every symbol the header declares, with (restype, argtypes)
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
SIGNATURES = {
    "tt_create": (ctypes.c_int, [_P, _I32, _P, _P, _I32, _I32, ctypes.POINTER(_P)]),
    "tt_create_ex": (ctypes.c_int, [_P, _I32, _P, _P, _I32, _I32, _P, ctypes.POINTER(_P)]),
    "tt_destroy": (None, [_P]),
    "tt_encode": (ctypes.c_int, [_P, _P, _I64, _P, ctypes.POINTER(_I64), _P]),
    "tt_encode_device": (ctypes.c_int, [_P, _P, _I64, _P, _P, _P]),
    "tt_encode_device_noalloc": (ctypes.c_int, [_P, _P, _I64, _P, _P, _P]),
    "tt_encode_batch": (ctypes.c_int, [_P, _P, _P, _I32, _P, _P, _P]),
    "tt_encode_spans": (ctypes.c_int, [_P, _P, _I64, _P, _P, ctypes.POINTER(_I64), _P]),
    "tt_encode_spans_device": (ctypes.c_int, [_P, _P, _I64, _P, _P, _P, _P]),
    "tt_pretokenize": (ctypes.c_int, [_P, _P, _I64, _P, ctypes.POINTER(_I64), _P]),
    "tt_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "tt_info": (ctypes.c_int, [_P, ctypes.POINTER(_I32), ctypes.POINTER(_I32), ctypes.POINTER(_I32)]),
    "tt_session_create": (ctypes.c_int, [_P, _I32, ctypes.POINTER(_P)]),
    "tt_session_destroy": (None, [_P]),
    "tt_session_append": (ctypes.c_int, [_P, _P, _I64, _P, _P]),
    "tt_session_tokens": (ctypes.c_int, [_P, _I64, _I64, _P, _P]),
    "tt_session_info": (ctypes.c_int, [_P, ctypes.POINTER(_I64), ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "tt_sync_boundaries": (ctypes.c_int, [_I32, _P, _I64, _P]),
    "tt_splice_plan": (ctypes.c_int, [_I32, _P, _I64, _I64, _I64, _P, _P, _I64, _P, _P, _I64, _I64,
                                      ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "tt_set_profiling": (ctypes.c_int, [_P, _I32]),
    "tt_stage_times": (ctypes.c_int, [_P, _P, _P, _I32, ctypes.POINTER(_I32)]),
}



class Options(ctypes.Structure):
    """``tt_options``: front-end options of ``tt_create_ex``."""

    _fields_ = [("ignore_merges", _I32), ("n_added", _I32), ("added_bytes", _P), ("added_offsets", _P),
                ("added_ids", _P)]


class AppendInfo(ctypes.Structure):
    """``tt_append_info``: the outcome of one session append."""

    _fields_ = [("kept", _I64), ("n_tokens", _I64), ("windows", _I32), ("full", _I32), ("window_chars", _I64)]


STAGES = ["tile"]  # TT_N_STAGES stages per call, in launch order

_lib = None


class TokTierError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        name = STATUS.get(status, str(status))
        super().__init__("%s%s (%s)" % (what + ": " if what else "", name, status))


def load():
    """The loaded library; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libtoktier.so is not built: run __graft_entry__.build() "
                              "or python -m paper_2607_29678_amd._build")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def check(status, what=""):
    if status != TT_OK:
        raise TokTierError(status, what)
