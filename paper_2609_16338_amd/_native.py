"""ctypes view of libbitcos.so (the C ABI in include/bitcos.h).

Loading fails loudly: there is no fallback implementation anywhere in this
package.  Build the library first (``python -m paper_2609_16338_amd.build_lib``).
"""

from __future__ import annotations

import ctypes
import os
import threading

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbitcos.so")

OK = 0
E_ARG = -1
E_VALUE = -2
E_SPACE = -3
E_HIP = -4
E_UNSUPPORTED = -5

FMT_BITCOS, FMT_TRIT5, FMT_BIT2 = 1, 2, 3
SEC_BITMAP, SEC_SIGNS, SEC_OFFSETS, SEC_SCALES = 0, 1, 2, 3
SEC_CODES = 0
X_I8, X_BF16 = 1, 2
Y_F32, Y_I32_RAW, Y_F32_ADD, Y_I32_RAW_ADD = 1, 2, 3, 4
MAX_M = 16  # most activation rows per GEMV call
NOALLOC_MAX_ROWS = 262144  # rows bitcos_pack_device_noalloc's fixed workspace holds
KERNEL_GENERAL, KERNEL_STREAMING, KERNEL_MATRIX, KERNEL_SMALL_BATCH, KERNEL_FIXED = 1, 2, 3, 4, 5
LAYOUT_VERSION = 1


class Layout(ctypes.Structure):
    _fields_ = [
        ("version", ctypes.c_uint32),
        ("format", ctypes.c_uint32),
        ("n", ctypes.c_int32),
        ("k", ctypes.c_int32),
        ("group", ctypes.c_int32),
        ("unit_rows", ctypes.c_int32),
        ("nnz", ctypes.c_uint64),
        ("sec_off", ctypes.c_uint64 * 4),
        ("sec_bytes", ctypes.c_uint64 * 4),
        ("total_bytes", ctypes.c_uint64),
        ("payload_bits", ctypes.c_uint64),
    ]

    def __repr__(self) -> str:
        return (f"Layout(format={self.format}, n={self.n}, k={self.k}, group={self.group}, "
                f"unit_rows={self.unit_rows}, nnz={self.nnz}, total_bytes={self.total_bytes}, "
                f"payload_bits={self.payload_bits})")


class LaunchInfo(ctypes.Structure):
    _fields_ = [
        ("per_lane", ctypes.c_int32),
        ("seg_lanes", ctypes.c_int32),
        ("rows_per_step", ctypes.c_int32),
        ("lanes_used", ctypes.c_int32),
        ("waves", ctypes.c_int64),
        ("workgroups", ctypes.c_int64),
        ("kernel", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class BitcosError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} ({status})")


_lib = None
_lock = threading.Lock()

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t
_LP = ctypes.POINTER(Layout)

SIGNATURES = {
    "bitcos_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "bitcos_version": (ctypes.c_uint32, []),
    "bitcos_plan": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _LP]),
    "bitcos_pack": (ctypes.c_int, [_P, _P, _LP, _P, _SZ]),
    "bitcos_unpack": (ctypes.c_int, [_LP, _P, _SZ, _P, _P]),
    "bitcos_gemv": (ctypes.c_int, [_LP, _P, _I32, _P, _I32, _P, _P, _I32, _P]),
    "trit5_plan": (ctypes.c_int, [_P, _I32, _I32, _I32, _LP]),
    "trit5_pack": (ctypes.c_int, [_P, _P, _LP, _P, _SZ]),
    "trit5_unpack": (ctypes.c_int, [_LP, _P, _SZ, _P, _P]),
    "trit5_gemv": (ctypes.c_int, [_LP, _P, _I32, _P, _I32, _P, _P, _I32, _P]),
    "bit2_plan": (ctypes.c_int, [_P, _I32, _I32, _I32, _LP]),
    "bit2_pack": (ctypes.c_int, [_P, _P, _LP, _P, _SZ]),
    "bit2_unpack": (ctypes.c_int, [_LP, _P, _SZ, _P, _P]),
    "bit2_gemv": (ctypes.c_int, [_LP, _P, _I32, _P, _I32, _P, _P, _I32, _P]),
    "bitcos_describe": (ctypes.c_int, [_LP, _I32, _I32, ctypes.POINTER(LaunchInfo)]),
    "bitcos_quantize_act": (ctypes.c_int, [_P, _I32, _I32, _P, _P, _P]),
    "bitcos_add_partials": (ctypes.c_int, [_P, _P, _I32, ctypes.c_int64, _P]),
    "bitcos_batch_bytes": (ctypes.c_size_t, [_I32]),
    "bitcos_batch_build": (ctypes.c_int, [_I32, _I32, _P, _P, _P, _P, _P, _I32, _I32, _P, _SZ]),
    "bitcos_gemv_batch": (ctypes.c_int, [_P, _P, _P]),
    "bitcos_plan_device_workspace": (ctypes.c_size_t, [_I32]),
    "bitcos_plan_device": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _SZ, _LP, _P]),
    "bitcos_pack_device": (ctypes.c_int, [_P, _P, _LP, _P, _SZ, _P, _SZ, _P]),
    "bitcos_pack_device_noalloc": (ctypes.c_int, [_P, _P, _I32, _I32, _I32, _I32, _LP, _P, _SZ, _P]),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"libbitcos.so not found at {LIB_PATH}; build it with "
                    "`python -m paper_2609_16338_amd.build_lib` (needs ROCm hipcc)")
            h = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(h, name)
                fn.restype = res
                fn.argtypes = args
            _lib = h
    return _lib


def strerror(status: int) -> str:
    try:
        return lib().bitcos_strerror(status).decode()
    except RuntimeError:
        return f"status {status}"


def check(status: int, where: str) -> None:
    if status != OK:
        raise BitcosError(status, where)
