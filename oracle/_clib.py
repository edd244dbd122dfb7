"""ctypes loader for the oracle's C weight generator.  TEST INFRASTRUCTURE ONLY."""
import ctypes
import os

import numpy as np

from .build_oracle import SO_PATH, build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(SO_PATH):
            build()
        L = ctypes.CDLL(SO_PATH)
        L.oracle_splitmix_output.restype = ctypes.c_uint64
        L.oracle_splitmix_output.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_stream_key.restype = ctypes.c_uint64
        L.oracle_stream_key.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int]
        for name, ptr in (("oracle_wgen_rows", ctypes.c_double), ("oracle_wgen_rows_f32", ctypes.c_float)):
            fn = getattr(L, name)
            fn.restype = None
            fn.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                           ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ptr)]
        _lib = L
    return _lib


def splitmix_output(seed: int, n: int) -> int:
    return int(lib().oracle_splitmix_output(seed & (2**64 - 1), n))


def wgen_rows(seed, tensor, layer, n_cols, row0, nrows, bf16, dtype=np.float64, out=None):
    """Rows [row0, row0+nrows) of the logical matrix (tensor, layer) with n_cols columns.

    `out` (fp64, C-contiguous, shape (nrows, n_cols)) is filled in place when given.
    """
    if dtype == np.float64:
        if out is None:
            out = np.empty((nrows, n_cols), dtype=np.float64)
        assert out.shape == (nrows, n_cols) and out.dtype == np.float64 and out.flags.c_contiguous
        lib().oracle_wgen_rows(seed, tensor, layer, n_cols, row0, nrows, int(bf16),
                               out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    else:
        out = np.empty((nrows, n_cols), dtype=np.float32)
        lib().oracle_wgen_rows_f32(seed, tensor, layer, n_cols, row0, nrows, int(bf16),
                                   out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
    return out
