"""ctypes view of ``librdfft.so``: the C ABI of include/rdfft.h, names unchanged.

Argument marshalling only.  Loading fails loudly when the library is missing; there
is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librdfft.so")

RDFFT_F32 = 0
RDFFT_BF16 = 1
RDFFT_F16 = 2

RDFFT_OK = 0
RDFFT_EINVAL = -1
RDFFT_EUNSUPPORTED = -2
RDFFT_ELAUNCH = -3
RDFFT_EDEVICE = -4

# every entry point include/rdfft.h declares
EXPORTS = (
    "rdfft_forward",
    "rdfft_inverse",
    "rdfft_pairs_to_halfcomplex",
    "rdfft_halfcomplex_to_pairs",
    "rdfft_forward_halfcomplex",
    "rdfft_inverse_halfcomplex",
    "bca_forward",
    "bca_backward",
    "bca_forward_batched",
    "bca_backward_batched",
    "rdfft_init",
    "rdfft_table_bytes",
    "rdfft_status_string",
)


class BcaGrads(ctypes.Structure):
    """bca_grads_t"""

    _fields_ = [("dx", ctypes.c_void_p), ("dc", ctypes.c_void_p)]


_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2511_01385_amd.build.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    for name in ("rdfft_forward", "rdfft_inverse", "rdfft_pairs_to_halfcomplex", "rdfft_halfcomplex_to_pairs",
                 "rdfft_forward_halfcomplex", "rdfft_inverse_halfcomplex"):
        f = getattr(lib, name)
        f.argtypes = [vp, i64, i64, i32, vp]
        f.restype = i32
    for name in ("bca_forward", "bca_backward"):
        f = getattr(lib, name)
        f.argtypes = [vp, vp, vp, ctypes.POINTER(BcaGrads), i64, i64, i64, i64, i32, vp]
        f.restype = i32
    pp = ctypes.POINTER(ctypes.c_void_p)
    lib.bca_forward_batched.argtypes = [i32, pp, pp, pp, i64, i64, i64, i64, i32, vp]
    lib.bca_forward_batched.restype = i32
    lib.bca_backward_batched.argtypes = [i32, pp, pp, pp, ctypes.POINTER(BcaGrads), i64, i64, i64, i64, i32, vp]
    lib.bca_backward_batched.restype = i32
    lib.rdfft_init.argtypes = []
    lib.rdfft_init.restype = i32
    lib.rdfft_table_bytes.argtypes = []
    lib.rdfft_table_bytes.restype = i64
    lib.rdfft_status_string.argtypes = [i32]
    lib.rdfft_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().rdfft_status_string(status).decode()
