"""ctypes declarations of liblcvq.so (the C ABI in include/lcvq.h)."""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblcvq.so")

# lcvq_status_t
OK, EINVAL, EUNSUPPORTED, EALIGN, EWORKSPACE, EHIP = range(6)
# lcvq_dtype_t
F32, BF16 = 0, 1
# lcvq_src_t
SRC_LATENT, SRC_CODES_U8, SRC_PACKED2 = 0, 1, 2
# lcvq_mask_t
MASK_ROUNDED, MASK_LATENT = 0, 1
# lcvq_op_t
OP_FWD, OP_BWD, OP_FWD_PACKED = 0, 1, 2
EST_STE, EST_DGE = 0, 1
# lcvq_kernel_t
KERNELS = ["fwd_prep", "fwd", "bwd_prep", "dx", "dw", "pack", "dequant", "fill", "adam", "packed_prep",
           "packed", "encode", "map_sum"]

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t

SIGNATURES = {
    "lcvq_pack2bit": (_I32, [_P, _I32, _I32, _I64, _I64, _P, _P]),
    "lcvq_dequant": (_I32, [_I64, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _I32, _P]),
    "lcvq_workspace_bytes": (_SZ, [_I32, _I64, _I64, _I64, _I32, _I32]),
    "lcvq_linear_fwd": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "lcvq_encode": (_I32, [_I64, _I64, _I32, _P, _I32, _P, _P, _P, _P, _P]),
    "lcvq_linear_fwd_ex": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, ctypes.c_float, ctypes.c_float, _P, _P, _P,
                                  _P, _P, _P, _SZ, _P]),
    "lcvq_linear_bwd_ex": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, ctypes.c_float, ctypes.c_float, _P, _P, _P,
                                  _P, _I32, _I32, ctypes.c_float, ctypes.c_float, _I32, _P, _P, _I32, _P, _P, _P,
                                  _SZ, _P]),
    "lcvq_saved_bytes": (_SZ, [_I64, _I64, _I64, _I32, _I32]),
    "lcvq_linear_fwd_train": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, ctypes.c_float, ctypes.c_float, _P, _P, _P,
                                     _P, _P, _P, _SZ, _P, _SZ, _P]),
    "lcvq_linear_bwd_train": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, ctypes.c_float, ctypes.c_float, _P, _P, _P,
                                     _P, _I32, _I32, ctypes.c_float, ctypes.c_float, _I32, _P, _P, _I32, _P, _P, _P,
                                     _SZ, _P, _SZ, _P]),
    "lcvq_linear_fwd_packed": (_I32, [_I64, _I64, _I64, _I32, _P, _P, _P, _P, _P, _I32, _P, _SZ, _P]),
    "lcvq_linear_fwd_packed_noalloc": (_I32, [_I64, _I64, _I64, _I32, _P, _P, _P, _P, _P, _I32, _P]),
    "lcvq_packed_scratch_bytes": (_SZ, []),
    "lcvq_linear_bwd": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, _P, _P, _P, _P, _I32, _I32,
                               _P, _P, _I32, _P, _P, _P, _SZ, _P]),
    "lcvq_linear_bwd_dge": (_I32, [_I64, _I64, _I64, _I32, _I32, _P, _P, _P, _P, _P, _I32, ctypes.c_float,
                                   ctypes.c_float, _I32, _P, _P, _I32, _P, _P, _P, _SZ, _P]),
    "lcvq_adamw_step": (_I32, [_P, _P, _I32, _P, _P, _P, _I32, _I64, ctypes.c_float, ctypes.c_float,
                                ctypes.c_float, ctypes.c_float, ctypes.c_float, _I32, _P]),
    "lcvq_xavier_quantizer": (_I32, [_I64, _I64, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float)]),
    "lcvq_xavier_init": (_I32, [_I64, _I64, _I32, _P, _P, _I32, _P]),
    "lcvq_timer_enable": (_I32, [ctypes.c_uint32]),
    "lcvq_timer_read": (_I32, [_I32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "lcvq_status_string": (ctypes.c_char_p, [_I32]),
    "lcvq_last_error": (ctypes.c_char_p, []),
}

_lib = None


class LcvqError(RuntimeError):
    """A non-OK status returned by liblcvq."""

    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: {status_string(status)} ({detail})")


def load() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2606_10531_amd.build.build() "
                               "(the LC-VQ layer has no non-HIP fallback)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    return load().lcvq_status_string(status).decode()


def last_error() -> str:
    return load().lcvq_last_error().decode()


def check(status: int, func: str) -> None:
    if status != OK:
        raise LcvqError(status, func, last_error())
