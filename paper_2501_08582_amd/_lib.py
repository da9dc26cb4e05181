"""ctypes binding of ``liblors.so`` (argument marshalling only).

Every function here forwards to the C ABI declared in ``include/lors.h`` and
turns a non-zero status into :class:`LorsError`.  There is no fallback: if the
library is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("LORS_LIBRARY", os.path.join(_PKG, "liblors.so"))

# lors_status_t
OK = 0
ERR_NULL = 1
ERR_DTYPE = 2
ERR_SHAPE = 3
ERR_MASK_FORMAT = 4
ERR_ALIGN = 5
ERR_ALIAS = 6
ERR_WORKSPACE = 7
ERR_UNSUPPORTED = 8
ERR_NOT_2_4 = 9
ERR_HIP = 10

DTYPE_BF16 = 0
DTYPE_F32 = 1
MASK_BITMAP = 0
MASK_2_4 = 1
FLAG_BWD_STE = 0x1
FLAG_REUSE_MASK_T = 0x2
FLAG_FWD_SPARSE_MFMA = 0x4
FLAG_SPLIT_LAST_WAVE = 0x8

EXPORTED = (
    "lors_status_string", "lors_version", "lors_mask_packed_bytes", "lors_mask_pack",
    "lors_mask_unpack", "lors_mask_from_weight", "lors_mask_pack_host", "lors_mask_unpack_host",
    "lors_workspace_bytes", "lors_forward", "lors_backward", "lors_backward_data",
    "lors_backward_weight", "lors_backward_noalloc",
)
NOALLOC_SCRATCH_BYTES = 32 << 20


class Problem(ctypes.Structure):
    _fields_ = [
        ("R", ctypes.c_int64),
        ("C", ctypes.c_int64),
        ("L", ctypes.c_int64),
        ("r", ctypes.c_int64),
        ("scale", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("mask_format", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
    ]


class LorsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {string(status)}")


_lib = None
_lock = threading.Lock()

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t


def _declare(lib) -> None:
    P = ctypes.POINTER(Problem)
    sig = {
        "lors_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "lors_version": (ctypes.c_int, []),
        "lors_mask_packed_bytes": (_sz, [_i64, _i64]),
        "lors_mask_pack": (ctypes.c_int, [_vp, _i64, _i64, _i32, _vp, _vp, _vp]),
        "lors_mask_unpack": (ctypes.c_int, [_vp, _i64, _i64, _i32, _vp, _vp]),
        "lors_mask_from_weight": (ctypes.c_int, [_vp, _i32, _i64, _i64, _i32, _vp, _vp, _vp]),
        "lors_mask_pack_host": (ctypes.c_int, [_vp, _i64, _i64, _i32, _vp, _vp]),
        "lors_mask_unpack_host": (ctypes.c_int, [_vp, _i64, _i64, _i32, _vp]),
        "lors_workspace_bytes": (_sz, [P]),
        "lors_forward": (ctypes.c_int, [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
        "lors_backward": (ctypes.c_int,
                          [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
        "lors_backward_data": (ctypes.c_int, [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
        "lors_backward_weight": (ctypes.c_int,
                                 [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
        "lors_backward_noalloc": (ctypes.c_int, [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def lib():
    """Load ``liblors.so`` once; raise if it is missing."""
    global _lib
    if _lib is None:
        with _lock:
            if _lib is None:
                if not os.path.exists(LIB_PATH):
                    raise RuntimeError(
                        f"{LIB_PATH} is missing: build it with "
                        "`python -m paper_2501_08582_amd.build` (hipcc, gfx950)")
                l = ctypes.CDLL(LIB_PATH)
                _declare(l)
                _lib = l
    return _lib


def string(status: int) -> str:
    return lib().lors_status_string(int(status)).decode()


def check(status: int, where: str) -> None:
    if status != OK:
        raise LorsError(status, where)


def problem(R, C, L, r, scale, dtype, mask_format, flags=0) -> Problem:
    return Problem(int(R), int(C), int(L), int(r), float(scale), int(dtype), int(mask_format),
                   int(flags))


# Thin pass-throughs (pointers are ints or None; stream is an int handle or None).
def mask_packed_bytes(R, C) -> int:
    return lib().lors_mask_packed_bytes(int(R), int(C))


def workspace_bytes(p: Problem) -> int:
    return lib().lors_workspace_bytes(ctypes.byref(p))


def mask_pack(dense, R, C, fmt, packed, first_bad, stream) -> int:
    return lib().lors_mask_pack(dense, R, C, fmt, packed, first_bad, stream)


def mask_unpack(packed, R, C, fmt, dense, stream) -> int:
    return lib().lors_mask_unpack(packed, R, C, fmt, dense, stream)


def mask_from_weight(W, dtype, R, C, fmt, packed, first_bad, stream) -> int:
    return lib().lors_mask_from_weight(W, dtype, R, C, fmt, packed, first_bad, stream)


def mask_pack_host(dense, R, C, fmt, packed, first_bad) -> int:
    return lib().lors_mask_pack_host(dense, R, C, fmt, packed, first_bad)


def mask_unpack_host(packed, R, C, fmt, dense) -> int:
    return lib().lors_mask_unpack_host(packed, R, C, fmt, dense)


def forward(p: Problem, X, W, M, B, A, bias, Y, ws, ws_bytes, stream) -> int:
    return lib().lors_forward(ctypes.byref(p), X, W, M, B, A, bias, Y, ws, ws_bytes, stream)


def backward(p: Problem, dY, X, W, M, B, A, dX, dB, dA, dbias, ws, ws_bytes, stream) -> int:
    return lib().lors_backward(ctypes.byref(p), dY, X, W, M, B, A, dX, dB, dA, dbias, ws,
                               ws_bytes, stream)


def backward_data(p: Problem, dY, W, M, B, A, dX, ws, ws_bytes, stream) -> int:
    return lib().lors_backward_data(ctypes.byref(p), dY, W, M, B, A, dX, ws, ws_bytes, stream)


def backward_weight(p: Problem, dY, X, M, B, A, dB, dA, dbias, ws, ws_bytes, stream) -> int:
    return lib().lors_backward_weight(ctypes.byref(p), dY, X, M, B, A, dB, dA, dbias, ws, ws_bytes,
                                      stream)


def backward_noalloc(p: Problem, dY, X, W, M, B, A, dX, dB, dA, dbias, stream) -> int:
    return lib().lors_backward_noalloc(ctypes.byref(p), dY, X, W, M, B, A, dX, dB, dA, dbias, stream)
