"""ctypes loader for libxdit.so (the HIP library built from csrc/).

The library is loaded from this package directory only; there is no fallback.
If it has not been built, loading raises XditError (build it with
``python -m paper_2411_01738_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(HERE, "libxdit.so")

# Status codes of include/xdit.h
XDIT_OK = 0
STATUS = {
    0: "XDIT_OK", -1: "XDIT_ERR_NULL", -2: "XDIT_ERR_DTYPE", -3: "XDIT_ERR_SHAPE",
    -4: "XDIT_ERR_RANGE", -5: "XDIT_ERR_LAYOUT", -6: "XDIT_ERR_ALIAS",
    -7: "XDIT_ERR_UNSUPPORTED", -8: "XDIT_ERR_HIP",
}
XDIT_BF16, XDIT_F32 = 0, 1
XDIT_MAX_PARTIALS = 64
XDIT_MAX_RANGES = 2
XDIT_MAX_SPLITS = 16

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32

SIGNATURES = {
    "xdit_patch_attn": (ctypes.c_int, [_vp, _vp, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _i64, _i64,
                                       _i32]),
    "xdit_patch_attn_ranges": (ctypes.c_int, [_vp, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                              _i64, _i64, _i64, _i64, _i32]),
    "xdit_chunk_attn": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i32]),
    "xdit_split_workspace_bytes": (_i64, [_i64, _i64, _i64, _i64, _i64, _i32, _i32]),
    "xdit_chunk_attn_split": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i64, _i64, _i64,
                                             _i64, _i64, _i64, _i32]),
    "xdit_chunk_attn_split_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _i64, _i64, _i64,
                                                     _i64, _i64, _i32]),
    "xdit_noalloc_scratch_bytes": (_i64, []),
    "xdit_patch_attn_split": (ctypes.c_int, [_vp, _i64, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                             _i32, _vp, _i64, _i64, _i64, _i64, _i64, _i32]),
    "xdit_chunk_attn_accum": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64,
                                             _i32]),
    "xdit_chunk_attn_accum_split": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _i64, _i64,
                                                   _i64, _i64, _i64, _i64, _i32]),
    "xdit_lse_merge": (ctypes.c_int, [_vp, _vp, _i32, _vp, _vp, _i64, _i64, _i64, _i64, _i32]),
    "xdit_kv_update": (ctypes.c_int, [_vp, _i64, _i64, _vp, _vp, _i64, _i64, _i64, _i64, _i32]),
    "xdit_stage_step": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp,
                                       _vp, _i64, _i64, _i64, _i64, _i64, _i32]),
    "xdit_set_stream": (ctypes.c_int, [_vp]),
    "xdit_get_stream": (_vp, []),
    "xdit_last_error": (ctypes.c_char_p, []),
    "xdit_version": (ctypes.c_char_p, []),
}


class XditError(RuntimeError):
    def __init__(self, code: int, message: str):
        self.code = code
        super().__init__(f"{STATUS.get(code, code)}: {message}")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library with argument types set (loaded once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            raise XditError(-8, f"{LIBRARY} is missing: build it with "
                                "`python -m paper_2411_01738_amd.build`")
        handle = ctypes.CDLL(LIBRARY)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def check(code: int) -> None:
    if code != XDIT_OK:
        raise XditError(code, lib().xdit_last_error().decode())
