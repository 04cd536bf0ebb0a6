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
_i16p = ctypes.POINTER(ctypes.c_int16)


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
        lib.oracle_f16_rne.argtypes = [ctypes.c_double]
        lib.oracle_f16_rne.restype = ctypes.c_uint16
        lib.oracle_f16_value.argtypes = [ctypes.c_uint16]
        lib.oracle_f16_value.restype = ctypes.c_double
        lib.oracle_f16_rne_array.argtypes = [_f64p, _u16p, ctypes.c_int64]
        lib.oracle_f16_rne_array.restype = None
        lib.oracle_split_f16.argtypes = [_f32p, _u16p, _u16p, ctypes.c_int64]
        lib.oracle_split_f16.restype = None
        lib.oracle_split_f16_range.argtypes = [ctypes.c_uint32, ctypes.c_int64, _u16p, _u16p]
        lib.oracle_split_f16_range.restype = None
        lib.oracle_f16_weight_exponent.argtypes = [ctypes.c_double]
        lib.oracle_f16_weight_exponent.restype = ctypes.c_int32
        lib.oracle_f16_weights.argtypes = [_f32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_int32, _u16p]
        lib.oracle_f16_weights.restype = None
        lib.oracle_gemm_f16w.argtypes = [ctypes.c_int] + [ctypes.c_int64] * 3 + [
            _f32p, ctypes.c_int64, _f32p, ctypes.c_int64, ctypes.c_int32, _i64p, ctypes.c_int64,
            _f64p, _f32p]
        lib.oracle_gemm_f16w.restype = ctypes.c_int
        lib.oracle_maxabs.argtypes = [_f32p, ctypes.c_int64]
        lib.oracle_maxabs.restype = ctypes.c_float
        lib.oracle_quantize_i16.argtypes = [_f32p, ctypes.c_int64, _i16p, _f32p]
        lib.oracle_quantize_i16.restype = None
        lib.oracle_unpack_i16_array.argtypes = [_i16p, _u16p, _u16p, ctypes.c_int64]
        lib.oracle_unpack_i16_array.restype = None
        lib.oracle_scores_i16.argtypes = [ctypes.c_int64] * 3 + [
            _i16p, ctypes.c_int64, _i16p, ctypes.c_int64, ctypes.c_float, ctypes.c_float,
            ctypes.c_float, _i64p, ctypes.c_int64, _f64p, _f32p]
        lib.oracle_scores_i16.restype = ctypes.c_int
        lib.oracle_scores_factor.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float]
        lib.oracle_scores_factor.restype = ctypes.c_double
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

    # ---- FP16 forms (HEAL-Base / HEAL-Full) and INT16 scores (HEAL+) ----

    def f16_rne(self, x):
        """binary16 bit patterns (uint16) of the float64 array ``x``, RNE."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        out = np.empty(x.shape, np.uint16)
        self.lib.oracle_f16_rne_array(_ptr(x, _f64p), _ptr(out, _u16p), x.size)
        return out

    def split_f16(self, x):
        """HEAL-Full pair (h_hi, h_lo) as binary16 bit patterns of float32 ``x``."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        hi = np.empty(x.shape, np.uint16)
        lo = np.empty(x.shape, np.uint16)
        self.lib.oracle_split_f16(_ptr(x, _f32p), _ptr(hi, _u16p), _ptr(lo, _u16p), x.size)
        return hi, lo

    def split_f16_range(self, start, n):
        hi = np.empty(n, np.uint16)
        lo = np.empty(n, np.uint16)
        self.lib.oracle_split_f16_range(start, n, _ptr(hi, _u16p), _ptr(lo, _u16p))
        return hi, lo

    def f16_weight_exponent(self, maxabs):
        return int(self.lib.oracle_f16_weight_exponent(float(maxabs)))

    def f16_weights(self, W, e):
        """RNE_f16(W * 2^e) bit patterns of the float32 N x K weight ``W``."""
        W = np.ascontiguousarray(W, dtype=np.float32)
        N, K = W.shape
        out = np.empty((N, K), np.uint16)
        if W.size:
            self.lib.oracle_f16_weights(_ptr(W, _f32p), N, K, max(K, 1), int(e), _ptr(out, _u16p))
        return out

    def gemm_f16w(self, A, W, e, products, rows=None):
        """HEAL-Base (products=1) / HEAL-Full (products=2) product A * W^T.

        A is float32 M x K, W the float32 weight N x K, e its exponent.
        Returns ``(C, S)`` as ``gemm3``.
        """
        A = np.ascontiguousarray(A, dtype=np.float32)
        W = np.ascontiguousarray(W, dtype=np.float32)
        assert A.ndim == 2 and W.ndim == 2 and A.shape[1] == W.shape[1]
        M, K = A.shape
        N = W.shape[0]
        rows_arr, n_out, rows_ptr = self._rows(rows, M)
        S = np.zeros((n_out, N), np.float64)
        C = np.zeros((n_out, N), np.float32)
        if n_out and N:
            rc = self.lib.oracle_gemm_f16w(products, M, N, K, _ptr(A, _f32p), max(K, 1),
                                           _ptr(W, _f32p), max(K, 1), int(e), rows_ptr, n_out,
                                           _ptr(S, _f64p), _ptr(C, _f32p))
            if rc != 0:
                raise ValueError("oracle_gemm_f16w failed")
        return C, S

    def maxabs(self, x):
        x = np.ascontiguousarray(x, dtype=np.float32).ravel()
        return np.float32(self.lib.oracle_maxabs(_ptr(x, _f32p), x.size))

    def quantize_i16(self, x):
        """(codes int16, max|x| float32) of the float32 tensor ``x``."""
        x = np.ascontiguousarray(x, dtype=np.float32)
        q = np.empty(x.shape, np.int16)
        m = np.zeros(1, np.float32)
        self.lib.oracle_quantize_i16(_ptr(x, _f32p), x.size, _ptr(q, _i16p), _ptr(m, _f32p))
        return q, m[0]

    def unpack_i16(self, q):
        q = np.ascontiguousarray(q, dtype=np.int16)
        hi = np.empty(q.shape, np.uint16)
        lo = np.empty(q.shape, np.uint16)
        self.lib.oracle_unpack_i16_array(_ptr(q, _i16p), _ptr(hi, _u16p), _ptr(lo, _u16p), q.size)
        return hi, lo

    def scores_factor(self, maxQ, maxK, alpha=1.0):
        """FP64 factor alpha (maxQ/32767)(maxK/32767) of the INT16 scores."""
        return float(self.lib.oracle_scores_factor(float(np.float32(maxQ)),
                                                   float(np.float32(maxK)),
                                                   float(np.float32(alpha))))

    def scores_i16(self, Q, Kt, maxQ, maxK, alpha=1.0, rows=None):
        """Dual-FP16 scores of INT16 Q (M x d) and K (N x d); ``(C, S)`` with S
        the integer dot products of the codes and C = f32(factor * S)."""
        Q = np.ascontiguousarray(Q, dtype=np.int16)
        Kt = np.ascontiguousarray(Kt, dtype=np.int16)
        assert Q.ndim == 2 and Kt.ndim == 2 and Q.shape[1] == Kt.shape[1]
        M, K = Q.shape
        N = Kt.shape[0]
        rows_arr, n_out, rows_ptr = self._rows(rows, M)
        S = np.zeros((n_out, N), np.float64)
        C = np.zeros((n_out, N), np.float32)
        if n_out and N:
            rc = self.lib.oracle_scores_i16(M, N, K, _ptr(Q, _i16p), max(K, 1), _ptr(Kt, _i16p),
                                            max(K, 1), float(np.float32(maxQ)),
                                            float(np.float32(maxK)), float(np.float32(alpha)),
                                            rows_ptr, n_out, _ptr(S, _f64p), _ptr(C, _f32p))
            if rc != 0:
                raise MemoryError("oracle_scores_i16 failed to allocate")
        return C, S

    @staticmethod
    def _rows(rows, M):
        if rows is None:
            return None, M, None
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        assert rows_arr.ndim == 1 and (rows_arr.size == 0 or
                                       (rows_arr.min() >= 0 and rows_arr.max() < M))
        return rows_arr, rows_arr.size, _ptr(rows_arr, _i64p)

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


def f16_bits_to_float(h):
    """Widen binary16 bit patterns (uint16) to float32 values."""
    return np.asarray(h, dtype=np.uint16).view(np.float16).astype(np.float32)


def bf16_bits_to_float(h):
    """Widen bf16 bit patterns (uint16) to float32 values."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
