"""ctypes binding of libsparseinfer.so: same names as include/sparseinfer.h.

Argument marshalling only.  The shared library is loaded on first use and a
missing library is an error (there is no fallback implementation).
"""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparseinfer.so")

SI_OK = 0
SI_ERR_NULL = 1
SI_ERR_SHAPE = 2
SI_ERR_ALIGN = 3
SI_ERR_ALPHA = 4
SI_ERR_WORKSPACE = 5
SI_ERR_HIP = 6
SI_ERR_FLAGS = 7
SI_ERR_ARG = 8
SI_ERR_TIMEOUT = 9
SI_ERR_LIST = 10
SI_NO_AS = 1
SI_NO_SPECULATION = 2

_p = ctypes.c_void_p
_i = ctypes.c_int
_sz = ctypes.c_size_t
_f = ctypes.c_float
_u32 = ctypes.c_uint32

# name -> (restype, argtypes)
SIGNATURES = {
    "si_last_error": (ctypes.c_char_p, []),
    "si_version": (ctypes.c_char_p, []),
    "si_signs_bytes": (_sz, [_i, _i]),
    "si_pack_signs": (_i, [_p, _i, _i, _p, _p]),
    "si_signs_to_canonical": (_i, [_p, _i, _i, _p, _p]),
    "si_transpose_down": (_i, [_p, _i, _i, _p, _p]),
    "si_alpha_threshold": (ctypes.c_int32, [_f, _i]),
    "si_workspace_bytes": (_sz, [_i, _i, _i]),
    "si_workspace_check": (_i, [_p, _sz, _p]),
    "si_device_error_status": (_i, [_u32]),
    "si_read_h3": (_i, [_p, _sz, _i, _i, _i, _p, _p, _p]),
    "si_read_bandwidth_probe": (_i, [_p, _sz, _p, _p]),
    "si_single_launch": (_i, [_i, _i, _i]),
    "si_predict": (_i, [_p, _i, _i, _p, _i, _f, _p, _p, _p, _p, _sz, _p]),
    "si_sparse_mlp": (_i, [_p, _p, _p, _i, _i, _p, _i, _p, _p, _p, _p, _p, _sz, _u32, _p, _p]),
    "si_predict_sparse_mlp": (_i, [_p, _p, _p, _p, _i, _i, _p, _i, _f, _p, _p, _p, _p, _p, _sz, _u32,
                                   _p, _p]),
    "si_predict_sparse_mlp_noalloc": (_i, [_p, _p, _p, _p, _i, _i, _p, _i, _f, _p, _p, _p, _p, _u32, _p, _p]),
    "si_sparse_relu_mlp": (_i, [_p, _p, _i, _i, _p, _i, _p, _p, _p, _p, _p, _sz, _u32, _p, _p]),
    "si_predict_sparse_relu_mlp": (_i, [_p, _p, _p, _i, _i, _p, _i, _f, _p, _p, _p, _p, _p, _sz, _u32,
                                        _p, _p]),
    "si_quantize_rows_i8": (_i, [_p, _i, _i, _p, _p, _p]),
    "si_pack_signs_i8": (_i, [_p, _i, _i, _p, _p]),
    "si_transpose_down_i8": (_i, [_p, _i, _i, _p, _p]),
    "si_sparse_mlp_i8": (_i, [_p, _p, _p, _p, _p, _p, _i, _i, _p, _i, _p, _p, _p, _sz, _u32, _p, _p]),
    "si_predict_sparse_mlp_i8": (_i, [_p, _p, _p, _p, _p, _p, _p, _i, _i, _p, _i, _f, _p, _p, _p, _p, _p, _sz,
                                      _u32, _p, _p]),
    "si_rmsnorm_predict_sparse_mlp": (_i, [_p, _p, _f, _p, _p, _p, _p, _i, _i, _i, _f, _p, _p, _p, _p, _p, _sz,
                                           _u32, _p, _p]),
}

_lib = None


class SparseInferError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


def load() -> ctypes.CDLL:
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2411_12692_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def call(name: str, *args) -> None:
    """Call an entry point that returns si_status; raise on failure."""
    lib = load()
    st = getattr(lib, name)(*args)
    if st != SI_OK:
        raise SparseInferError(st, lib.si_last_error().decode())


def status(name: str, *args) -> int:
    """Call an entry point and return its raw status (no exception)."""
    return getattr(load(), name)(*args)


def last_error() -> str:
    return load().si_last_error().decode()
