"""ctypes loader for libisoquant.so (the C ABI in include/isoquant.h).

Loading never falls back to anything: if the shared library has not been
built, every entry point raises.
"""

from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
# IQ_LIB_PATH selects another build of the same library (e.g. the
# host-sanitized one of build.py); there is no fallback either way
LIB_PATH = os.environ.get("IQ_LIB_PATH") or os.path.join(_PKG, "libisoquant.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "isoquant.h")

IQ_OK = 0
STATUS_NAMES = {
    0: "IQ_OK",
    1: "IQ_ERR_INVALID_ARGUMENT",
    2: "IQ_ERR_UNSUPPORTED",
    3: "IQ_ERR_WORKSPACE_TOO_SMALL",
    4: "IQ_ERR_HIP",
    5: "IQ_ERR_CAPACITY",
}
IQ_DTYPE_F32 = 0
IQ_DTYPE_F16 = 1

_c_i64 = ctypes.c_int64
_c_u64 = ctypes.c_uint64
_c_int = ctypes.c_int
_vp = ctypes.c_void_p
_c_size = ctypes.c_size_t
_c_float = ctypes.c_float

class IqCodebook(ctypes.Structure):
    """iq_codebook_t: bits, then the first 2^bits levels and 2^bits - 1
    thresholds of fixed-size arrays."""
    _fields_ = [("bits", ctypes.c_int32), ("levels", ctypes.c_float * 16),
                ("thresholds", ctypes.c_float * 15)]


_cbp = ctypes.POINTER(IqCodebook)

_SIGNATURES = {
    "iq_status_string": (ctypes.c_char_p, [_c_int]),
    "iq_version": (_c_int, []),
    "iq_codebook": (_c_int, [_vp, _vp]),
    "iq_make_rotation": (_c_int, [_c_u64, _c_i64, _c_i64, _vp]),
    "iq_make_rotation_variant": (_c_int, [_c_u64, _c_i64, _c_i64, _c_int, _vp]),
    "iq_fit_rotation": (_c_int, [_vp, _c_i64, _c_i64, _c_i64, _c_int, _vp]),
    "iq_compress_kv_paged": (_c_int, [_vp, _vp, _c_int, _c_i64, _c_i64, _c_i64, _c_i64, _vp,
                                      _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp, _c_i64,
                                      _c_i64, _vp]),
    "iq_decode_attention_paged": (_c_int, [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp,
                                           _c_i64, _vp, _c_i64, _vp, _c_i64, _c_i64, _c_i64,
                                           _c_i64, _c_float, _vp, _vp, _c_size, _vp]),
    "iq_decode_step_paged": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _c_i64,
                                      _c_i64, _vp, _c_i64, _vp, _c_i64, _vp, _c_i64, _c_i64,
                                      _c_i64, _c_i64, _c_float, _vp, _vp, _c_size, _vp, _vp]),
    "iq_so4_to_quaternions": (_c_int, [_vp, _vp]),
    "iq_codebook_bits": (_c_int, [_c_int, _vp, _vp]),
    "iq_decode_step_bits": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp, _c_i64,
                                     _c_i64, _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_float, _vp,
                                     _vp, _c_size, _vp, _c_int, _vp]),
    "iq_decode_multi_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                                  _c_i64]),
    "iq_decode_attention_multi": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp,
                                           _c_i64, _c_i64, _c_i64, _c_i64, _c_i64, _c_float,
                                           _vp, _vp, _c_size, _vp]),
    "iq_decode_attention_multi_bits": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64,
                                                _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                                _c_float, _vp, _vp, _c_size, _c_int, _vp]),
    "iq_decode_step_multi": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp, _c_i64,
                                      _c_i64, _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                      _c_float, _vp, _vp, _c_size, _vp, _c_int, _vp]),
    "iq_decode_attention_multi_paged": (_c_int, [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp,
                                                 _c_i64, _vp, _c_i64, _vp, _c_i64, _c_i64,
                                                 _c_i64, _c_i64, _c_i64, _c_float, _vp, _vp,
                                                 _c_size, _vp]),
    "iq_compress_kv_bits": (_c_int, [_vp, _vp, _c_int, _c_i64, _c_i64, _c_i64, _c_i64, _vp,
                                     _vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_int, _vp]),
    "iq_decode_attention_bits": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp,
                                          _c_i64, _c_i64, _c_i64, _c_i64, _c_float, _vp, _vp,
                                          _c_size, _c_int, _vp]),
    "iq_compress_kv": (_c_int, [_vp, _vp, _c_int, _c_i64, _c_i64, _c_i64, _c_i64, _vp,
                                _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp]),
    "iq_append_token": (_c_int, [_vp, _vp, _c_int, _c_i64, _c_i64, _c_i64, _vp,
                                 _vp, _vp, _vp, _vp, _c_i64, _vp, _vp, _vp]),
    "iq_decode_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i64, _c_i64, _c_i64]),
    "iq_decode_workspace_init": (_c_int, [_vp, _c_size, _vp]),
    "iq_decode_attention": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp,
                                     _c_i64, _c_i64, _c_i64, _c_i64, _c_float, _vp, _vp,
                                     _c_size, _vp]),
    "iq_decode_step": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp, _c_i64,
                                _c_i64, _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_float, _vp,
                                _vp, _c_size, _vp, _vp]),
    "iq_dequantize_kv": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_i64,
                                  _c_i64, _c_i64, _c_i64, _c_int, _vp, _vp, _vp]),
    "iq_decode_f16_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i64, _c_i64, _c_i64]),
    "iq_decode_attention_f16": (_c_int, [_vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_i64, _c_i64,
                                         _c_i64, _c_i64, _c_float, _vp, _vp, _c_size, _vp]),
    "iq_decode_step_noalloc": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp,
                                        _c_i64, _c_i64, _vp, _c_i64, _c_i64, _c_i64, _c_i64,
                                        _c_float, _vp, _vp, _vp]),
    "iq_decode_attention_rope": (_c_int, [_vp, _vp, _vp, _vp, _vp, _c_i64, _vp, _vp, _vp, _c_i64,
                                          _c_i64, _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                          _c_float, _vp, _vp, _c_size, _vp]),
    "iq_fit_codebook": (_c_int, [_vp, _c_i64, _c_i64, _c_i64, _vp, ctypes.c_int32, _cbp]),
    "iq_compress_kv_cb": (_c_int, [_vp, _vp, _c_int, _c_i64, _c_i64, _c_i64, _c_i64, _vp, _cbp,
                                   _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp]),
    "iq_decode_attention_cb": (_c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _vp, _cbp,
                                        _c_i64, _c_i64, _c_i64, _c_i64, _c_float, _vp, _vp,
                                        _c_size, _vp]),
    "iq_decode_step_cb": (_c_int, [_vp, _vp, _vp, _c_int, _vp, _vp, _vp, _vp, _vp, _c_i64,
                                   _c_i64, _vp, _cbp, _c_i64, _c_i64, _c_i64, _c_i64, _c_float,
                                   _vp, _vp, _c_size, _vp, _vp]),
    "iq_dequantize_kv_cb": (_c_int, [_vp, _vp, _vp, _vp, _vp, _cbp, _vp, _c_i64, _c_i64, _c_i64,
                                     _c_i64, _c_i64, _c_i64, _c_int, _vp, _vp, _vp]),
    "iq_stream_read_sink_words": (_c_size, [_c_size, ctypes.c_int32, ctypes.c_int32]),
    "iq_stream_read": (_c_int, [_vp, _c_size, _vp, _c_size, ctypes.c_int32, ctypes.c_int32,
                                ctypes.c_uint32, _vp]),
}

_lib = None


class IsoQuantError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {STATUS_NAMES.get(status, status)}")


def lib() -> ctypes.CDLL:
    """The loaded library (loaded once).  Raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                "(python -m paper_2608_08081_amd.build)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def check(fn: str, status: int) -> None:
    if status != IQ_OK:
        raise IsoQuantError(fn, status)


def header_functions() -> list[str]:
    """Names of the functions declared in include/isoquant.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(iq_[a-z0-9_]+)\s*\(", text)))
