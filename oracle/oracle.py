"""ctypes wrapper around the CPU oracle (test infrastructure only).

``Oracle(path)`` loads a built oracle library; the module-level helpers use
the default ``oracle/liboracle.so``, building it first if it is absent.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _ptr(a, t):
    return a.ctypes.data_as(t)


class Oracle:
    """The oracle functions of one built library."""

    def __init__(self, path):
        lib = ctypes.CDLL(path)
        lib.oracle_bf16_rne.argtypes = [ctypes.c_float]
        lib.oracle_bf16_rne.restype = ctypes.c_uint16
        lib.oracle_split.argtypes = [_f32p, _u16p, _u16p, ctypes.c_int64]
        lib.oracle_split.restype = None
        lib.oracle_split_range.argtypes = [ctypes.c_uint32, ctypes.c_int64, _u16p, _u16p]
        lib.oracle_split_range.restype = None
        lib.oracle_gemm3.argtypes = [ctypes.c_int64] * 3 + [_f32p, ctypes.c_int64, _f32p,
                                                            ctypes.c_int64, ctypes.c_float,
                                                            _i64p, ctypes.c_int64, _f64p, _f32p]
        lib.oracle_gemm3.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def split(self, x):
        """(hi, lo) bf16 bit patterns (uint16) of the float32 array ``x``."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        hi = np.empty(x.shape, np.uint16)
        lo = np.empty(x.shape, np.uint16)
        self.lib.oracle_split(_ptr(x, _f32p), _ptr(hi, _u16p), _ptr(lo, _u16p), x.size)
        return hi, lo

    def split_range(self, start, n):
        """Split every FP32 bit pattern in [start, start + n)."""
        hi = np.empty(n, np.uint16)
        lo = np.empty(n, np.uint16)
        self.lib.oracle_split_range(start, n, _ptr(hi, _u16p), _ptr(lo, _u16p))
        return hi, lo

    def gemm3(self, A, B, alpha=1.0, rows=None):
        """Compensated product of row-major float32 A (M x K) and B (K x N).

        Returns ``(C, S)``: the FP32 result and the FP64 sum it was rounded
        from, for all rows, or for the listed ``rows`` of A in that order.
        """
        A = np.asarray(A, dtype=np.float32)
        B = np.asarray(B, dtype=np.float32)
        assert A.ndim == 2 and B.ndim == 2 and A.shape[1] == B.shape[0]
        if A.strides[1] != 4:
            A = np.ascontiguousarray(A)
        if B.strides[1] != 4:
            B = np.ascontiguousarray(B)
        M, K = A.shape
        N = B.shape[1]
        lda = A.strides[0] // 4 if M > 1 else max(K, 1)
        ldb = B.strides[0] // 4 if K > 1 else max(N, 1)
        if rows is None:
            rows_arr, n_out, rows_ptr = None, M, None
        else:
            rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
            assert rows_arr.ndim == 1 and (rows_arr.size == 0 or
                                           (rows_arr.min() >= 0 and rows_arr.max() < M))
            n_out, rows_ptr = rows_arr.size, _ptr(rows_arr, _i64p)
        S = np.zeros((n_out, N), np.float64)
        C = np.zeros((n_out, N), np.float32)
        if n_out and N:
            rc = self.lib.oracle_gemm3(M, N, K, _ptr(A, _f32p), lda, _ptr(B, _f32p), ldb,
                                       float(np.float32(alpha)), rows_ptr, n_out,
                                       _ptr(S, _f64p), _ptr(C, _f32p))
            if rc != 0:
                raise MemoryError("oracle_gemm3 failed to allocate")
        return C, S

    def num_threads(self):
        return self.lib.oracle_num_threads()


_default = None


def default():
    """The oracle built from ``oracle/heal_oracle.c`` (built if missing)."""
    global _default
    if _default is None:
        if not os.path.exists(_build.LIBRARY):
            _build.build()
        _default = Oracle(_build.LIBRARY)
    return _default


def bf16_bits_to_float(h):
    """Widen bf16 bit patterns (uint16) to float32 values."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
