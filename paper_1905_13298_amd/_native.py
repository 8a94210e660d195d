"""ctypes binding of ``libdeepshift.so`` (the C ABI declared in include/deepshift.h).

The functions keep the C names and arguments; they only convert Python values
to C types and turn a non-zero status into ``DeepShiftError``. Loading builds
the library first when it has not been built yet.
"""
from __future__ import annotations

import ctypes
import os
import threading

from . import build as _build

_lock = threading.Lock()
_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_U32 = ctypes.c_uint32

SIGNATURES = {
    "ds_packed_row_words": (_I64, [_I64]),
    "ds_pack_shift_weights": (ctypes.c_int, [_P, _I64, _I64, _P, _I64]),
    "ds_unpack_shift_weights": (ctypes.c_int, [_P, _I64, _I64, _P, _I64]),
    "ds_packed_row_words_bits": (_I64, [_I64, _I32]),
    "ds_pack_shift_weights_bits": (ctypes.c_int, [_P, _I64, _I64, _I32, _P, _I64]),
    "ds_unpack_shift_weights_bits": (ctypes.c_int, [_P, _I64, _I64, _I32, _P, _I64]),
    "ds_linear_shift": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I64, _I64, _I32, _U32, _P]),
    "ds_conv2d_shift": (ctypes.c_int, [_P, _P, _P, _P] + [_I64] * 7 + [_I32] * 4 + [_I32, _U32, _P]),
    "ds_conv2d_mul_i32": (ctypes.c_int, [_P, _P, _P, _P] + [_I64] * 7 + [_I32] * 4 + [_U32, _P]),
    "ds_linear_mul_i32": (ctypes.c_int, [_P, _P, _P, _P, _I64, _I64, _I64, _U32, _P]),
    "ds_conv2d_shift_describe": (ctypes.c_int, [_I64] * 7 + [_I32] * 4 + [ctypes.c_char_p, _I64]),
    "ds_quantize_shift_weights_q": (ctypes.c_int, [_P, _I64, _I64, _I32, _P, _U32, _P]),
    "ds_quantize_shift_weights_ps": (ctypes.c_int, [_P, _P, _I64, _I64, _I32, _P, _U32, _P]),
    "ds_quantize_shift_weights_q_many": (ctypes.c_int, [_I64, _P, _P, _P, _I32, _P, _U32, _P]),
    "ds_to_fixed_point": (ctypes.c_int, [_P, _I64, _I32, _P, _U32, _P]),
    "ds_conv2d_shift_fused": (ctypes.c_int, [_P, _P, _P, _P, _P, _I32, _P, _P] + [_I64] * 7 + [_I32] * 4 + [_I32, _U32, _P]),
    "ds_maxpool2d": (ctypes.c_int, [_P, _P] + [_I64] * 6 + [_I32] * 4 + [_U32, _P]),
    "ds_avgpool2d_global": (ctypes.c_int, [_P, _P] + [_I64] * 4 + [_U32, _P]),
    "ds_jit_conv_create": (ctypes.c_int, [_P, _P, _P, _P, _I32] + [_I64] * 7 + [_I32] * 4 + [_U32, _I32, _P]),
    "ds_jit_conv_run": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "ds_jit_conv_destroy": (ctypes.c_int, [_P]),
    "ds_jit_conv_image": (ctypes.c_int, [_P, _P, _P, _P, _I32] + [_I64] * 7 + [_I32] * 4 + [_U32, _I32, _P, _I64, _P]),
    "ds_jit_conv_query": (ctypes.c_int, [_P, _P, _P, _P]),
    "ds_jit_conv_layout": (ctypes.c_int, [_P, _P, _P, _P, _P, _P]),
    "ds_jit_conv_mul_create": (ctypes.c_int, [_P, _P] + [_I64] * 7 + [_I32] * 4 + [_U32, _I32, _P]),
    "ds_jit_conv_mul_image": (ctypes.c_int, [_P, _P] + [_I64] * 7 + [_I32] * 4 + [_U32, _I32, _P, _I64, _P]),
    "ds_jit_conv_backward_data_create": (ctypes.c_int, [_P] + [_I64] * 7 + [_I32] * 4 + [_U32, _I32, _P]),
    "ds_conv2d_shift_backward_data": (ctypes.c_int, [_P, _P, _P] + [_I64] * 7 + [_I32] * 4 + [_I32, _U32, _P]),
    "ds_linear_shift_backward_data": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I64, _I32, _U32, _P]),
    "ds_conv2d_shift_backward_data_describe": (ctypes.c_int, [_I64] * 7 + [_I32] * 4 + [ctypes.c_char_p, _I64]),
    "ds_conv2d_shift_noalloc": (ctypes.c_int, [_P, _P, _P, _P] + [_I64] * 7 + [_I32] * 4 + [_I32, _U32, _P]),
    "ds_conv2d_shift_noalloc_scratch_bytes": (_I64, [_I64] * 7 + [_I32] * 4),
    "ds_set_tuning": (ctypes.c_int, [ctypes.c_char_p, _I32]),
    "ds_get_tuning": (ctypes.c_int, [ctypes.c_char_p, _P]),
    "ds_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "ds_last_error_message": (ctypes.c_char_p, []),
}

STATUS = {
    0: "DS_SUCCESS", 1: "DS_ERR_NULL_POINTER", 2: "DS_ERR_INVALID_SHAPE",
    3: "DS_ERR_INVALID_ARG", 4: "DS_ERR_BUFFER_TOO_SMALL", 5: "DS_ERR_INVALID_CODE",
    6: "DS_ERR_HIP", 7: "DS_ERR_UNSUPPORTED",
}


class DeepShiftError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


def library_path() -> str:
    return _build.LIB


def lib():
    """The loaded library (built on first use when no build exists)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_build.LIB):
                _build.build()
            handle = ctypes.CDLL(_build.LIB)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
    return _lib


def check(status: int) -> None:
    if status != 0:
        msg = lib().ds_last_error_message().decode()
        raise DeepShiftError(status, msg)


def call(name: str, *args) -> None:
    """Call a status-returning entry point and raise on failure."""
    check(getattr(lib(), name)(*args))
