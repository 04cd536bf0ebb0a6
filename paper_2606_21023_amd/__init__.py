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
  lib()                               -> the raw ctypes library
"""
import ctypes
import os

__all__ = ["HealError", "lib", "library_path", "heal_split_f32", "heal_gemm_f32",
           "heal_gemm_f32_strided_batched", "heal_gemm_f32_instance", "select_instance",
           "INSTANCE_AUTO", "INSTANCE_LARGE", "INSTANCE_MEDIUM", "INSTANCE_SKINNY", "STATUS"]

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
    _lib = L
    return L


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
    if t.numel() and t.stride(-1) != 1:
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
