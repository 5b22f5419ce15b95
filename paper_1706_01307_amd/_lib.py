"""ctypes binding of libspconv.so (the C ABI declared in include/spconv.h).

Argument marshalling only: every step of the rule-book build and of the
forward runs in the library's HIP kernels.  PyTorch provides device memory
and the current stream.  There is no fallback: if the library is missing or
the device is not a GPU, calls raise.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspconv.so")

OK, EINVAL, EDUP, ERANGE, ENOMEM, ECAP, EHIP, ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7
VSC, SC = 0, 1
OP_VSC, OP_SC, OP_DC = 0, 1, 2
POOL_MAX, POOL_AVG = 0, 1
F32, BF16 = 0, 1
BUILD_ASYNC, BUILD_TRANSPOSE = 1, 2

# Every symbol the header declares, with its ctypes signature.
_P, _I, _I64, _U = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint
ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
RELEASE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p)

SIGNATURES = {
    "spconv_set_allocator": (_I, [ALLOC_FN, RELEASE_FN, _P]),
    "spconv_build_rulebook": (_I, [_I, _I, _P, _I64, _P, _P, _P, _U, _P, ctypes.POINTER(_P)]),
    "spconv_build_rulebook_on": (_I, [_P, _I, _P, _P, _U, _P, ctypes.POINTER(_P)]),
    "spconv_rulebook_bounds": (_I, [_P, _P, _P]),
    "spconv_release_cached_memory": (_I, [_P]),
    "spconv_memory_stats": (_I, [_I, _P, _P]),
    "spconv_rulebook_status": (_I, [_P]),
    "spconv_rulebook_query": (_I, [_P, _P, _P, _P, _P, _P]),
    "spconv_rulebook_export": (_I, [_P, _P, _P, _P]),
    "spconv_rulebook_out_coords": (_I, [_P, ctypes.POINTER(_P)]),
    "spconv_vsc_forward": (_I, [_P, _I, _P, _P, _P, _I, _P, _I, _I, _P]),
    "spconv_sc_forward": (_I, [_P, _I, _P, _P, _P, _I, _P, _I, _I, _P]),
    "spconv_forward_fused": (_I, [_P, _I, _P, _P, _P, _P, _P, _I, _I, _P, _I, _I, _P]),
    "spconv_pool_forward": (_I, [_P, _I, _I, _P, _P, _I, _P]),
    "spconv_dc_forward": (_I, [_P, _I, _P, _P, _P, _I, _P, _I, _I, _P]),
    "spconv_backward_data": (_I, [_P, _I, _I, _P, _P, _I, _P, _I, _I, _P]),
    "spconv_backward_weight_workspace": (_I, [_P, _I, _I, _I, ctypes.POINTER(ctypes.c_size_t)]),
    "spconv_backward_weight": (_I, [_P, _I, _I, _P, _P, _P, _P, _I, _I, _P, ctypes.c_size_t, _P]),
    "spconv_backward_weight_noalloc": (_I, [_P, _I, _I, _P, _P, _P, _P, _I, _I, _P]),
    "spconv_rulebook_destroy": (None, [_P]),
    "spconv_status_string": (ctypes.c_char_p, [_I]),
}


class SpconvError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        msg = _lib.spconv_status_string(status).decode() if _lib else str(status)
        super().__init__(f"{what}: {msg} ({status})" if what else f"{msg} ({status})")


_lib = None


def load():
    """Load libspconv.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it first (python -m paper_1706_01307_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def check(status, what=""):
    if status != OK:
        raise SpconvError(status, what)
