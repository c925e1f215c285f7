"""ctypes loader for libscanweaver.so (the C ABI declared in include/scanweaver.h).

The library is built in place by ``paper_2606_00601_amd.build``.  There is no
fallback: if it is missing, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libscanweaver.so")

SW_OK = 0
SW_ERR_INVALID_ARG = 1
SW_ERR_UNSUPPORTED = 2
SW_ERR_HIP = 3
SW_ERR_ALLOC = 4
SW_DTYPE_F32 = 0
SW_DTYPE_BF16 = 1
SW_DELTA_SOFTPLUS = 1
SW_SCHED_DEFAULT = 0
SW_SCHED_BLELLOCH = 1

# name -> (restype, argtypes), mirroring include/scanweaver.h
_vp, _i64, _int = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
SIGNATURES = {
    "sw_version": (_int, []),
    "sw_affine_scan": (_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64]),
    "sw_affine_scan_i32": (_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64]),
    "sw_affine_scan_noalloc": (_int, [_vp, _vp, _vp, _vp, _i64, _i64, _i64]),
    "sw_affine_scan_schedule": (_int, [_vp] * 4 + [_i64] * 3 + [_int]),
    "sw_selective_scan_fwd_schedule": (_int, [_vp] * 8 + [_i64] * 4 + [_int] * 2),
    "sw_affine_scan_schedule_i32": (_int, [_vp] * 4 + [_i64] * 3 + [_int]),
    "sw_affine_scan_proj": (_int, [_vp] * 7 + [_i64] * 3),
    "sw_selective_scan_bwd": (_int, [_vp] * 22 + [_i64] * 4 + [_int] * 3),
    "sw_selective_scan_fwd_train": (_int, [_vp] * 13 + [_i64] * 4 + [_int] * 3),
    "sw_selective_scan_plan": (_int, [_i64] * 4 + [_int] * 4 + [_vp] * 4),
    "sw_affine_scan_proj_i32": (_int, [_vp] * 7 + [_i64] * 3),
    "sw_selective_scan_fwd": (_int, [_vp] * 8 + [_i64] * 4),
    "sw_selective_scan_fwd_bf16": (_int, [_vp] * 8 + [_i64] * 4),
    "sw_selective_scan_fwd_ex": (_int, [_vp] * 11 + [_i64] * 4 + [_int] * 3),
    "sw_set_stream": (_int, [_vp]),
    "sw_get_stream": (_vp, []),
    "sw_status_string": (ctypes.c_char_p, [_int]),
    "sw_last_error": (ctypes.c_char_p, []),
    "sw_last_launch": (ctypes.c_char_p, []),
}

_lock = threading.Lock()
_lib = None


class ScanWeaverError(RuntimeError):
    """A non-OK status returned by libscanweaver."""

    def __init__(self, status: int, where: str, message: str):
        self.status = status
        super().__init__(f"{where}: {message} ({status_string(status)})")


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2606_00601_amd.build`")
            handle = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
        return _lib


_fast = None


def fast():
    """The extension module the binding calls the library through: one
    function per entry point with the same name and arguments as ``lib()``'s
    (addresses as ints or None), at a fraction of ctypes' per-call cost.
    It links the same libscanweaver.so, so the per-thread stream and error
    message are shared with ``lib()``.  Raises if it has not been built."""
    global _fast
    if _fast is not None:
        return _fast
    lib()
    try:
        from . import _swcall
    except ImportError as e:
        raise RuntimeError(f"the call extension is missing ({e}): build it with "
                           "`python -m paper_2606_00601_amd.build`") from e
    _fast = _swcall
    return _fast


def status_string(status: int) -> str:
    return lib().sw_status_string(int(status)).decode()


def last_error() -> str:
    return lib().sw_last_error().decode()


def check(status: int, where: str) -> None:
    if status != SW_OK:
        raise ScanWeaverError(status, where, last_error())
