"""HEAL compensated GEMM for MI355X: Python binding of ``libheal.so``.

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI declared in ``include/heal.h``.  PyTorch supplies
device memory and the current stream; nothing here computes on the host.
If the library is not built (``python -m paper_2606_21023_amd.build``), every
call raises ``HealError``: there is no fallback path.

Functions (names follow the C ABI):
  heal_split_f32(x)                   -> (hi, lo) bf16 bit patterns, torch.uint16
  heal_gemm_f32(A, B, out=None)       -> C = A @ B, bf16x3 compensated, FP32
  heal_gemm_f32_strided_batched(A, B, alpha=1.0, trans_b=False, out=None)
  heal_gemm_f32_instance(instance, A, B, ...)  -- a forced kernel instance
  heal_split_f16(x)                   -> (hi, lo) binary16 bit patterns (HEAL-Full pair)
  heal_maxabs_f32(x)                  -> max|x| as a 1-element float32 CUDA tensor
  heal_f16_weight_exponent(maxabs)    -> int e (host)
  heal_pack_f16_weight(W, e)          -> packed FP16 weight (torch.uint16)
  heal_gemm_f16w(A, W16, N, e, products)  -> HEAL-Base (1) / HEAL-Full (2) GEMM, FP32
  heal_presplit_b(B, trans_b=False)   -> packed bf16 (hi, lo) operand
  heal_gemm_f32_presplit(A, Bp, N)    -> bitwise equal to heal_gemm_f32(A, B)
  heal_quantize_i16(x)                -> (codes int16, max|x| 1-element tensor)
  heal_scores_i16(Q, Kt, maxQ, maxK, alpha)  -> dual-FP16 scores of INT16 codes, FP32
  lib()                               -> the raw ctypes library
  build_id(), check_build()           -> the library's source hash; refuse a stale binary
"""
import ctypes
import os

__all__ = ["HealError", "lib", "library_path", "build_id", "check_build", "heal_split_f32", "heal_gemm_f32",
           "heal_gemm_f32_strided_batched", "heal_gemm_f32_instance", "select_instance",
           "INSTANCE_AUTO", "INSTANCE_LARGE", "INSTANCE_MEDIUM", "INSTANCE_SKINNY", "STATUS",
           "heal_split_f16", "heal_packed_size", "heal_maxabs_f32", "heal_f16_weight_exponent",
           "heal_pack_f16_weight", "heal_gemm_f16w", "heal_presplit_b", "heal_gemm_f32_presplit",
           "heal_quantize_i16", "heal_scores_i16"]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libheal.so")

INSTANCE_AUTO, INSTANCE_LARGE, INSTANCE_MEDIUM, INSTANCE_SKINNY = 0, 1, 2, 3
STATUS = {0: "HEAL_OK", 1: "HEAL_ERR_INVALID_VALUE", 2: "HEAL_ERR_UNSUPPORTED_DEVICE",
          3: "HEAL_ERR_LAUNCH"}


class HealError(RuntimeError):
    """A libheal call failed, or the library is missing."""

    def __init__(self, msg, status=None):
        super().__init__(msg)
        self.status = status


_lib = None
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


def lib():
    """Load ``libheal.so`` (once) and declare its C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(library_path):
        raise HealError("libheal.so is not built (expected at %s); run "
                        "`python -m paper_2606_21023_amd.build`" % library_path)
    L = ctypes.CDLL(library_path)
    L.heal_status_string.argtypes = [ctypes.c_int]
    L.heal_status_string.restype = ctypes.c_char_p
    L.heal_version.argtypes = []
    L.heal_version.restype = ctypes.c_int
    L.heal_build_id.argtypes = []
    L.heal_build_id.restype = ctypes.c_char_p
    L.heal_split_f32.argtypes = [_vp, _vp, _vp, _i64, _vp]
    L.heal_split_f32.restype = ctypes.c_int
    L.heal_gemm_f32.argtypes = [_i64, _i64, _i64, _vp, _vp, _vp, _i64, _i64, _i64, _vp]
    L.heal_gemm_f32.restype = ctypes.c_int
    L.heal_gemm_f32_strided_batched.argtypes = [_i64, _i64, _i64, ctypes.c_float,
                                                _vp, _i64, _i64, _vp, _i64, _i64, ctypes.c_int,
                                                _vp, _i64, _i64, _i64, _vp]
    L.heal_gemm_f32_strided_batched.restype = ctypes.c_int
    L.heal_gemm_f32_instance.argtypes = [ctypes.c_int] + L.heal_gemm_f32_strided_batched.argtypes
    L.heal_gemm_f32_instance.restype = ctypes.c_int
    L.heal_gemm_select_instance.argtypes = [_i64, _i64]
    L.heal_gemm_select_instance.restype = ctypes.c_int
    _c = ctypes.c_int
    L.heal_split_f16.argtypes = [_vp, _vp, _vp, _i64, _vp]
    L.heal_split_f16.restype = _c
    L.heal_packed_size.argtypes = [_i64, _i64, _c]
    L.heal_packed_size.restype = _i64
    L.heal_maxabs_f32.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp]
    L.heal_maxabs_f32.restype = _c
    L.heal_f16_weight_exponent.argtypes = [ctypes.c_float, ctypes.POINTER(ctypes.c_int32)]
    L.heal_f16_weight_exponent.restype = _c
    L.heal_pack_f16_weight.argtypes = [_vp, _i64, _i64, _i64, ctypes.c_int32, _vp, _vp]
    L.heal_pack_f16_weight.restype = _c
    L.heal_gemm_f16w.argtypes = [_c, _i64, _i64, _i64, _vp, _i64, _vp, ctypes.c_int32, _vp, _i64,
                                 _vp]
    L.heal_gemm_f16w.restype = _c
    L.heal_gemm_f16w_instance.argtypes = [_c] + L.heal_gemm_f16w.argtypes
    L.heal_gemm_f16w_instance.restype = _c
    L.heal_presplit_b.argtypes = [_vp, _i64, _i64, _i64, _c, _vp, _vp]
    L.heal_presplit_b.restype = _c
    L.heal_gemm_f32_presplit.argtypes = [_i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp]
    L.heal_gemm_f32_presplit.restype = _c
    L.heal_gemm_f32_presplit_instance.argtypes = [_c] + L.heal_gemm_f32_presplit.argtypes
    L.heal_gemm_f32_presplit_instance.restype = _c
    L.heal_quantize_i16.argtypes = [_vp, _i64, _vp, _vp, _vp]
    L.heal_quantize_i16.restype = _c
    L.heal_scores_i16.argtypes = [_i64, _i64, _i64, _vp, _i64, _i64, _vp, _vp, _i64, _i64, _vp,
                                  ctypes.c_float, _vp, _i64, _i64, _i64, _vp]
    L.heal_scores_i16.restype = _c
    _lib = L
    return L


def build_id():
    """The source hash the loaded ``libheal.so`` was built from."""
    return lib().heal_build_id().decode()


def check_build():
    """Raise ``HealError`` unless the loaded ``libheal.so`` was built from the
    sources beside it (a stale binary would test old code)."""
    from . import build as _build
    want, got = _build.source_hash(), build_id()
    if got != want:
        raise HealError("libheal.so was built from other sources (build id %s, sources %s); "
                        "rebuild with `python -m paper_2606_21023_amd.build`" % (got, want))
    return got


def _check(status, what):
    if status != 0:
        raise HealError("%s failed: %s" % (what, STATUS.get(status, status)), status)


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _require(t, name, ndim):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise HealError("%s must be a CUDA (HIP) tensor" % name)
    if t.dtype != torch.float32:
        raise HealError("%s must be float32, got %s" % (name, t.dtype))
    if t.dim() != ndim:
        raise HealError("%s must have %d dimensions, got %d" % (name, ndim, t.dim()))
    if t.numel() and t.size(-1) > 1 and t.stride(-1) != 1:
        # (a last dimension of one element has no stride to respect: torch
        # may report any, e.g. for the transpose of a one-row matrix)
        raise HealError("%s must be contiguous in its last dimension" % name)


def _ld(t):
    """Row stride of the last two dims, in elements."""
    return t.stride(-2) if t.size(-2) > 1 else max(t.size(-1), 1)


def heal_split_f32(x, hi=None, lo=None):
    """Split a contiguous float32 CUDA tensor into bf16 (hi, lo) bit patterns."""
    import torch
    if not isinstance(x, torch.Tensor) or not x.is_cuda or x.dtype != torch.float32:
        raise HealError("x must be a float32 CUDA tensor")
    if not x.is_contiguous():
        raise HealError("x must be contiguous")
    if hi is None:
        hi = torch.empty(x.shape, dtype=torch.uint16, device=x.device)
    if lo is None:
        lo = torch.empty(x.shape, dtype=torch.uint16, device=x.device)
    _check(lib().heal_split_f32(x.data_ptr(), hi.data_ptr(), lo.data_ptr(), x.numel(), _stream()),
           "heal_split_f32")
    return hi, lo


def heal_gemm_f32(A, B, out=None):
    """C = A @ B (A: M x K, B: K x N, row-major float32 CUDA tensors)."""
    import torch
    _require(A, "A", 2)
    _require(B, "B", 2)
    M, K = A.shape
    if B.shape[0] != K:
        raise HealError("inner dimensions differ: %s @ %s" % (tuple(A.shape), tuple(B.shape)))
    N = B.shape[1]
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    _require(C, "out", 2)
    if tuple(C.shape) != (M, N):
        raise HealError("out has shape %s, expected %s" % (tuple(C.shape), (M, N)))
    _check(lib().heal_gemm_f32(M, N, K, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                               _ld(A), _ld(B), _ld(C), _stream()), "heal_gemm_f32")
    return C


def _batched(fn_args_prefix, A, B, alpha, trans_b, out, what):
    import torch
    _require(A, "A", 3)
    _require(B, "B", 3)
    bat, M, K = A.shape
    if trans_b:
        N, Kb = B.shape[1], B.shape[2]
    else:
        Kb, N = B.shape[1], B.shape[2]
    if Kb != K or B.shape[0] != bat:
        raise HealError("shapes do not match: A %s, B %s, trans_b=%s"
                        % (tuple(A.shape), tuple(B.shape), trans_b))
    C = out if out is not None else torch.empty((bat, M, N), dtype=torch.float32, device=A.device)
    _require(C, "out", 3)
    if tuple(C.shape) != (bat, M, N):
        raise HealError("out has shape %s, expected %s" % (tuple(C.shape), (bat, M, N)))
    sA = A.stride(0) if bat > 1 else 0
    sB = B.stride(0) if bat > 1 else 0
    sC = C.stride(0) if bat > 1 else 0
    st = fn_args_prefix(M, N, K, ctypes.c_float(alpha), A.data_ptr(), _ld(A), sA,
                        B.data_ptr(), _ld(B), sB, 1 if trans_b else 0,
                        C.data_ptr(), _ld(C), sC, bat, _stream())
    _check(st, what)
    return C


def heal_gemm_f32_strided_batched(A, B, alpha=1.0, trans_b=False, out=None):
    """C[b] = alpha * A[b] @ op(B[b]) for 3-D tensors; op(B) = B^T if trans_b."""
    return _batched(lib().heal_gemm_f32_strided_batched, A, B, alpha, trans_b, out,
                    "heal_gemm_f32_strided_batched")


def heal_gemm_f32_instance(instance, A, B, alpha=1.0, trans_b=False, out=None):
    """As heal_gemm_f32_strided_batched with a forced kernel instance (2-D or 3-D)."""
    squeeze = A.dim() == 2
    if squeeze:
        A, B = A.unsqueeze(0), B.unsqueeze(0)
        out = out.unsqueeze(0) if out is not None else None
    f = lib().heal_gemm_f32_instance
    C = _batched(lambda *a: f(int(instance), *a), A, B, alpha, trans_b, out,
                 "heal_gemm_f32_instance")
    return C[0] if squeeze else C


def select_instance(M, N):
    """The instance heal_gemm_f32 chooses for an M x N output."""
    return lib().heal_gemm_select_instance(M, N)


# ---- FP16 forms, pre-split operand, INT16 scores ---------------------------

def _require_dtype(t, name, dtype, ndim=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise HealError("%s must be a CUDA (HIP) tensor" % name)
    if t.dtype != dtype:
        raise HealError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if ndim is not None and t.dim() != ndim:
        raise HealError("%s must have %d dimensions, got %d" % (name, ndim, t.dim()))
    if t.numel() and t.size(-1) > 1 and t.stride(-1) != 1:
        # (a last dimension of one element has no stride to respect: torch
        # may report any, e.g. for the transpose of a one-row matrix)
        raise HealError("%s must be contiguous in its last dimension" % name)


def heal_split_f16(x, hi=None, lo=None):
    """HEAL-Full pair of a contiguous float32 CUDA tensor, binary16 bit patterns."""
    import torch
    _require_dtype(x, "x", torch.float32)
    if not x.is_contiguous():
        raise HealError("x must be contiguous")
    if hi is None:
        hi = torch.empty(x.shape, dtype=torch.uint16, device=x.device)
    if lo is None:
        lo = torch.empty(x.shape, dtype=torch.uint16, device=x.device)
    _check(lib().heal_split_f16(x.data_ptr(), hi.data_ptr(), lo.data_ptr(), x.numel(), _stream()),
           "heal_split_f16")
    return hi, lo


def heal_packed_size(K, N, planes):
    n = lib().heal_packed_size(K, N, planes)
    if n < 0:
        raise HealError("invalid packed size K=%d N=%d planes=%d" % (K, N, planes))
    return n


def heal_maxabs_f32(x, out=None):
    """max|x| of a 2-D (or contiguous) float32 CUDA tensor, as a 1-element tensor."""
    import torch
    _require_dtype(x, "x", torch.float32)
    if x.dim() == 2:
        rows, cols, ld = x.shape[0], x.shape[1], _ld(x)
    else:
        if not x.is_contiguous():
            raise HealError("x must be 2-D or contiguous")
        rows, cols, ld = 1, x.numel(), max(x.numel(), 1)
    out = out if out is not None else torch.empty(1, dtype=torch.float32, device=x.device)
    _check(lib().heal_maxabs_f32(x.data_ptr(), rows, cols, ld, out.data_ptr(), _stream()),
           "heal_maxabs_f32")
    return out


def heal_f16_weight_exponent(maxabs):
    """Largest e with maxabs * 2^e <= 65504 (host)."""
    e = ctypes.c_int32()
    _check(lib().heal_f16_weight_exponent(ctypes.c_float(float(maxabs)), ctypes.byref(e)),
           "heal_f16_weight_exponent")
    return e.value


def heal_pack_f16_weight(W, e, out=None):
    """Packed RNE_f16(W * 2^e) of an N x K float32 weight (torch.uint16, 1-D)."""
    import torch
    _require_dtype(W, "W", torch.float32, 2)
    N, K = W.shape
    size = heal_packed_size(K, N, 1)
    out = out if out is not None else torch.empty(size, dtype=torch.uint16, device=W.device)
    _check(lib().heal_pack_f16_weight(W.data_ptr(), N, K, _ld(W), int(e), out.data_ptr(),
                                      _stream()), "heal_pack_f16_weight")
    return out


def heal_gemm_f16w(A, W16, N, e, products, out=None, instance=INSTANCE_AUTO):
    """HEAL-Base (products=1) or HEAL-Full (products=2): A (M x K float32) times
    the packed FP16 weight of an N x K matrix, scaled back by 2^-e."""
    import torch
    _require_dtype(A, "A", torch.float32, 2)
    M, K = A.shape
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    _require_dtype(C, "out", torch.float32, 2)
    if tuple(C.shape) != (M, N):
        raise HealError("out has shape %s, expected %s" % (tuple(C.shape), (M, N)))
    if W16.numel() < heal_packed_size(K, N, 1):
        raise HealError("W16 is smaller than the packed size")
    _check(lib().heal_gemm_f16w_instance(int(instance), int(products), M, N, K, A.data_ptr(),
                                         _ld(A), W16.data_ptr(), int(e), C.data_ptr(), _ld(C),
                                         _stream()), "heal_gemm_f16w")
    return C


def heal_presplit_b(B, trans_b=False, out=None):
    """Packed bf16 (hi, lo) of B (K x N, or N x K with trans_b)."""
    import torch
    _require_dtype(B, "B", torch.float32, 2)
    K, N = (B.shape[1], B.shape[0]) if trans_b else (B.shape[0], B.shape[1])
    size = heal_packed_size(K, N, 2)
    out = out if out is not None else torch.empty(size, dtype=torch.uint16, device=B.device)
    _check(lib().heal_presplit_b(B.data_ptr(), K, N, _ld(B), 1 if trans_b else 0,
                                 out.data_ptr(), _stream()), "heal_presplit_b")
    return out


def heal_gemm_f32_presplit(A, Bp, N, out=None, instance=INSTANCE_AUTO):
    """C = A @ B from the pre-split packed B of an operand with N columns."""
    import torch
    _require_dtype(A, "A", torch.float32, 2)
    M, K = A.shape
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    _require_dtype(C, "out", torch.float32, 2)
    if tuple(C.shape) != (M, N):
        raise HealError("out has shape %s, expected %s" % (tuple(C.shape), (M, N)))
    if Bp.numel() < heal_packed_size(K, N, 2):
        raise HealError("Bp is smaller than the packed size")
    _check(lib().heal_gemm_f32_presplit_instance(int(instance), M, N, K, A.data_ptr(), _ld(A),
                                                 Bp.data_ptr(), C.data_ptr(), _ld(C), _stream()),
           "heal_gemm_f32_presplit")
    return C


def heal_quantize_i16(x, q=None, maxabs=None):
    """INT16 codes of a contiguous float32 CUDA tensor and its max|x| (device)."""
    import torch
    _require_dtype(x, "x", torch.float32)
    if not x.is_contiguous():
        raise HealError("x must be contiguous")
    q = q if q is not None else torch.empty(x.shape, dtype=torch.int16, device=x.device)
    maxabs = maxabs if maxabs is not None else torch.empty(1, dtype=torch.float32,
                                                           device=x.device)
    _check(lib().heal_quantize_i16(x.data_ptr(), x.numel(), q.data_ptr(), maxabs.data_ptr(),
                                   _stream()), "heal_quantize_i16")
    return q, maxabs


def heal_scores_i16(Q, Kt, maxQ, maxK, alpha=1.0, out=None):
    """Scores of INT16 codes: Q (batch x M x d), Kt (batch x N x d) -> batch x M x N
    FP32 (2-D inputs give a 2-D result)."""
    import torch
    squeeze = Q.dim() == 2
    if squeeze:
        Q, Kt = Q.unsqueeze(0), Kt.unsqueeze(0)
        out = out.unsqueeze(0) if out is not None else None
    _require_dtype(Q, "Q", torch.int16, 3)
    _require_dtype(Kt, "Kt", torch.int16, 3)
    bat, M, K = Q.shape
    N = Kt.shape[1]
    if Kt.shape[0] != bat or Kt.shape[2] != K:
        raise HealError("shapes do not match: Q %s, Kt %s" % (tuple(Q.shape), tuple(Kt.shape)))
    S = out if out is not None else torch.empty((bat, M, N), dtype=torch.float32, device=Q.device)
    _require_dtype(S, "out", torch.float32, 3)
    sQ = Q.stride(0) if bat > 1 else 0
    sK = Kt.stride(0) if bat > 1 else 0
    sS = S.stride(0) if bat > 1 else 0
    _check(lib().heal_scores_i16(M, N, K, Q.data_ptr(), _ld(Q), sQ, maxQ.data_ptr(),
                                 Kt.data_ptr(), _ld(Kt), sK, maxK.data_ptr(),
                                 ctypes.c_float(alpha), S.data_ptr(), _ld(S), sS, bat,
                                 _stream()), "heal_scores_i16")
    return S[0] if squeeze else S
