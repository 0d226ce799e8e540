"""ctypes loader for libacdc.so (the HIP library built in-tree).

Fails loudly when the library is missing: there is no CPU fallback.
"""

from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libacdc.so")

_lib = None

# Exported symbols and their signatures (mirrors include/acdc.h).
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_U32 = ctypes.c_uint32
_SZ = ctypes.c_size_t
SIGNATURES = {
    "acdc_supported": (ctypes.c_int, [_I32, _U32]),
    "acdc_prepare": (ctypes.c_int, [_I32, _U32]),
    "acdc_saved_bytes": (_SZ, [_I64, _I32, _I32, _U32]),
    "acdc_forward_workspace_size": (_SZ, [_I64, _I32, _I32, _U32]),
    "acdc_backward_workspace_size": (_SZ, [_I64, _I32, _I32, _U32, ctypes.c_int]),
    "acdc_forward": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _I64, _I32, _I32, _U32, _P, _SZ, _P, _SZ, _P]),
    "acdc_forward_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _I64, _I32, _I32, _U32, _P, _SZ, _P]),
    "acdc_backward": (ctypes.c_int,
                      [_P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P, _P, _P, _I64, _I32, _I32, _U32, _P, _SZ, _P]),
    "acdc_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "acdc_profile_read": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "acdc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "acdc_last_hip_error": (ctypes.c_int, []),
    "acdc_sync_timeouts": (ctypes.c_int, [ctypes.POINTER(ctypes.c_int64), ctypes.c_int]),
}


class LibraryMissing(RuntimeError):
    pass


def lib():
    """The loaded library (loaded once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(
                f"{LIB_PATH} is not built; run `python -m paper_1511_05946_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(rc: int) -> str:
    return lib().acdc_status_string(int(rc)).decode()
