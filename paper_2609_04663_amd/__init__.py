"""Python binding of libemu: FP32/FP64 GEMM emulated through BF16 component
products on AMD Instinct MI355X (gfx950), after arxiv 2609.04663.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libemu.so`` (C ABI in ``include/emu.h``).  PyTorch supplies the
device memory and the stream; tensors must be CUDA (HIP) tensors, row-major
with unit stride in the last dimension.  There is no CPU fallback: if the
library is not built, importing the functions raises.

    sgemm(A, B, C=None)            -> C = A @ B, FP32, 3 components / 6 products
    dgemm(A, B, nprod, C=None)     -> C = A @ B, FP64, six slices / nprod products
    sgemm_ex / dgemm_ex(..., transa, transb, alpha, beta) -> BLAS form alpha op(A) op(B) + beta C
    split_f32(X, as_b=False)       -> int16 tensor [3, R, C] of BF16 bit patterns
    split_f64(X, as_b=False)       -> (int16 tensor [6, R, C], int32 tensor [6])
    set_split_scope(scope)         -> SCOPE_OPERAND (default) or SCOPE_ROWCOL weights
    scale_exponents(X, by_col)     -> int32 tensor of the ROWCOL weights
    domain_status()                -> EMU_STATUS_* bits accumulated since last call
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libemu.so")

EMU_OK, EMU_EINVAL, EMU_EHIP, EMU_ENOMEM = 0, 1, 2, 3
STATUS_NAN, STATUS_RANGE, STATUS_SUBNORMAL, STATUS_OVERFLOW, STATUS_INEXACT = 1, 2, 4, 8, 16
STATUS_FALLBACK = 32
FALLBACK_NONE, FALLBACK_FP64 = 0, 1
SGEMM_SPLIT_PASS, SGEMM_SPLIT_STREAMED = 0, 1
SPLIT_SYM, SPLIT_LITERAL = 0, 1
SCOPE_OPERAND, SCOPE_ROWCOL, SCOPE_KBIN = 0, 1, 2
# the paper's product counts N_p(d), d = 3 .. 6 (Eq. fp64productcounts) ...
NPROD = (6, 10, 15, 21)
# ... and every depth d = 1 .. 11 of the selection S_d (Eq. product-selection)
NPROD_ALL = (1, 3, 6, 10, 15, 21, 26, 30, 33, 35, 36)

EXPORTS = ("emu_sgemm", "emu_dgemm", "emu_set_stream", "emu_set_split_mode",
           "emu_domain_status", "emu_last_error", "emu_release_workspace",
           "emu_workspace_bytes", "emu_split_f32", "emu_split_f64", "emu_profile_enable",
           "emu_profile_read", "emu_set_split_scope", "emu_scale_exponents", "emu_sgemm_ex",
           "emu_dgemm_ex", "emu_dgemm_noalloc", "emu_set_fallback", "emu_set_sgemm_split")


class EmuError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libemu error {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libemu.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2609_04663_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i64, p, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        L.emu_sgemm.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64]
        L.emu_dgemm.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, ci]
        L.emu_dgemm_noalloc.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, ci]
        L.emu_set_stream.argtypes = [p]
        L.emu_set_split_mode.argtypes = [ci]
        L.emu_set_split_scope.argtypes = [ci]
        L.emu_set_fallback.argtypes = [ci]
        L.emu_set_sgemm_split.argtypes = [ci]
        ch, f32, f64 = ctypes.c_char, ctypes.c_float, ctypes.c_double
        L.emu_sgemm_ex.argtypes = [ch, ch, i64, i64, i64, f32, p, i64, p, i64, f32, p, i64]
        L.emu_dgemm_ex.argtypes = [ch, ch, i64, i64, i64, f64, p, i64, p, i64, f64, p, i64, ci]
        L.emu_scale_exponents.argtypes = [i64, i64, p, i64, ci, p]
        L.emu_domain_status.argtypes = [ctypes.POINTER(ctypes.c_uint)]
        L.emu_last_error.restype = ctypes.c_char_p
        L.emu_workspace_bytes.restype = i64
        L.emu_split_f32.argtypes = [i64, i64, p, i64, ci, p]
        L.emu_split_f64.argtypes = [i64, i64, p, i64, ci, p, p]
        L.emu_profile_enable.argtypes = [ci]
        L.emu_profile_read.argtypes = [i64, p, p, ctypes.POINTER(ctypes.c_int64)]
        for name in ("emu_sgemm", "emu_dgemm", "emu_set_stream", "emu_set_split_mode",
                     "emu_domain_status", "emu_release_workspace", "emu_split_f32",
                     "emu_split_f64", "emu_profile_enable", "emu_profile_read",
                     "emu_set_split_scope", "emu_scale_exponents", "emu_sgemm_ex",
                     "emu_dgemm_ex", "emu_dgemm_noalloc", "emu_set_fallback",
                     "emu_set_sgemm_split"):
            getattr(L, name).restype = ci
        _lib = L
    return _lib


def _check(rc: int):
    if rc != EMU_OK:
        raise EmuError(rc, lib().emu_last_error().decode())


def _bind_stream(dev: torch.device):
    lib().emu_set_stream(ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))


def _layout(t: torch.Tensor, dtype, name: str):
    """dtype and row-major layout checks (metadata only, any device)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    # the stride of a dimension of extent 1 is never used (NumPy-made tensors
    # of shape (1, n) can carry a row stride of 1)
    if (t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1)
            or (t.shape[0] > 1 and t.stride(0) < max(1, t.shape[1]))):
        raise ValueError(f"{name} must be a row-major 2-D tensor with unit column stride")
    return t


def _on_gpu(*named):
    for name, t in named:
        if not t.is_cuda:
            raise TypeError(f"{name} must be a GPU tensor")


def _mat(t: torch.Tensor, dtype, name: str):
    _layout(t, dtype, name)
    _on_gpu((name, t))
    return t


def _out(C, M: int, N: int, dtype, device):
    """The output C: allocated when None, else checked to be M x N (the
    library writes M rows of ldc elements: a smaller C would be overrun)."""
    if C is None:
        return torch.empty((M, N), dtype=dtype, device=device)
    _layout(C, dtype, "C")
    if tuple(C.shape) != (M, N):
        raise ValueError(f"C must be {M} x {N}, got {tuple(C.shape)}")
    return C


def _ld(t: torch.Tensor) -> int:
    if t.shape[0] <= 1:
        return max(1, t.shape[1])
    return max(1, t.stride(0), t.shape[1])


def sgemm(A: torch.Tensor, B: torch.Tensor, C: torch.Tensor | None = None) -> torch.Tensor:
    _layout(A, torch.float32, "A")
    _layout(B, torch.float32, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    C = _out(C, M, N, torch.float32, A.device)
    _on_gpu(("A", A), ("B", B), ("C", C))
    _bind_stream(A.device)
    _check(lib().emu_sgemm(M, N, K, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), C.data_ptr(),
                           _ld(C)))
    return C


def dgemm(A: torch.Tensor, B: torch.Tensor, nprod: int,
          C: torch.Tensor | None = None) -> torch.Tensor:
    _layout(A, torch.float64, "A")
    _layout(B, torch.float64, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    C = _out(C, M, N, torch.float64, A.device)
    _on_gpu(("A", A), ("B", B), ("C", C))
    _bind_stream(A.device)
    _check(lib().emu_dgemm(M, N, K, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B), C.data_ptr(),
                           _ld(C), int(nprod)))
    return C


def dgemm_noalloc(A: torch.Tensor, B: torch.Tensor, nprod: int, C: torch.Tensor) -> torch.Tensor:
    """dgemm into a caller-supplied C without any device allocation by the
    library (its fixed scratch; see emu_dgemm_noalloc in emu.h)."""
    _layout(A, torch.float64, "A")
    _layout(B, torch.float64, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    if C is None:
        raise ValueError("dgemm_noalloc needs C")
    C = _out(C, M, N, torch.float64, A.device)
    _on_gpu(("A", A), ("B", B), ("C", C))
    _bind_stream(A.device)
    _check(lib().emu_dgemm_noalloc(M, N, K, A.data_ptr(), _ld(A), B.data_ptr(), _ld(B),
                                   C.data_ptr(), _ld(C), int(nprod)))
    return C


def _op_shape(X: torch.Tensor, trans: str):
    if trans not in ("N", "T"):
        raise ValueError("trans must be 'N' or 'T'")
    return (X.shape[1], X.shape[0]) if trans == "T" else tuple(X.shape)


def _gemm_ex(fn, dtype, A, B, C, transa, transb, alpha, beta, extra=()):
    _layout(A, dtype, "A")
    _layout(B, dtype, "B")
    M, K = _op_shape(A, transa)
    K2, N = _op_shape(B, transb)
    if K != K2:
        raise ValueError("inner dimensions differ")
    if C is None and beta != 0:
        raise ValueError("beta != 0 needs C")
    C = _out(C, M, N, dtype, A.device)
    _on_gpu(("A", A), ("B", B), ("C", C))
    _bind_stream(A.device)
    _check(fn(transa.encode(), transb.encode(), M, N, K, alpha, A.data_ptr(), _ld(A),
              B.data_ptr(), _ld(B), beta, C.data_ptr(), _ld(C), *extra))
    return C


def sgemm_ex(A, B, C=None, transa="N", transb="N", alpha=1.0, beta=0.0):
    """C = alpha op(A) op(B) + beta C in FP32 (A, B as stored; see emu.h)."""
    return _gemm_ex(lib().emu_sgemm_ex, torch.float32, A, B, C, transa, transb, float(alpha),
                    float(beta))


def dgemm_ex(A, B, nprod, C=None, transa="N", transb="N", alpha=1.0, beta=0.0):
    """C = alpha op(A) op(B) + beta C in FP64 with nprod retained products."""
    return _gemm_ex(lib().emu_dgemm_ex, torch.float64, A, B, C, transa, transb, float(alpha),
                    float(beta), (int(nprod),))


def split_f32(X: torch.Tensor, as_b: bool = False) -> torch.Tensor:
    _mat(X, torch.float32, "X")
    R, Cc = X.shape
    out = torch.empty((3, R, Cc), dtype=torch.int16, device=X.device)
    _bind_stream(X.device)
    _check(lib().emu_split_f32(R, Cc, X.data_ptr(), _ld(X), int(as_b), out.data_ptr()))
    return out


def split_f64(X: torch.Tensor, as_b: bool = False):
    _mat(X, torch.float64, "X")
    R, Cc = X.shape
    out = torch.empty((6, R, Cc), dtype=torch.int16, device=X.device)
    v = torch.empty(6, dtype=torch.int32, device=X.device)
    _bind_stream(X.device)
    _check(lib().emu_split_f64(R, Cc, X.data_ptr(), _ld(X), int(as_b), out.data_ptr(),
                               v.data_ptr()))
    return out, v


def set_split_mode(mode: int):
    _check(lib().emu_set_split_mode(int(mode)))


def set_sgemm_split(mode: int):
    """SGEMM_SPLIT_PASS (split kernel, then the product kernel) or
    SGEMM_SPLIT_STREAMED (the product kernel splits its own k-blocks)."""
    _check(lib().emu_set_sgemm_split(int(mode)))


def set_fallback(mode: int):
    """FALLBACK_NONE (the paper's behaviour) or FALLBACK_FP64 (see emu.h)."""
    _check(lib().emu_set_fallback(int(mode)))


def set_split_scope(scope: int):
    """SCOPE_OPERAND (the paper's split) or SCOPE_ROWCOL (row/column weights)."""
    _check(lib().emu_set_split_scope(int(scope)))


def scale_exponents(X: torch.Tensor, by_col: bool = False) -> torch.Tensor:
    _mat(X, torch.float64, "X")
    R, Cc = X.shape
    out = torch.empty(Cc if by_col else R, dtype=torch.int32, device=X.device)
    _bind_stream(X.device)
    _check(lib().emu_scale_exponents(R, Cc, X.data_ptr(), _ld(X), int(by_col), out.data_ptr()))
    return out


def domain_status() -> int:
    f = ctypes.c_uint(0)
    _check(lib().emu_domain_status(ctypes.byref(f)))
    return int(f.value)


def profile_enable(on: bool = True):
    """Record split/pack and GEMM phase times of every call (see emu.h)."""
    _check(lib().emu_profile_enable(int(on)))


def profile_read(cap: int = 4096):
    """Per-call (split_ms, gemm_ms) lists of the profiled calls since the last
    read, oldest first; synchronises."""
    s = (ctypes.c_double * cap)()
    g = (ctypes.c_double * cap)()
    n = ctypes.c_int64()
    _check(lib().emu_profile_read(cap, s, g, ctypes.byref(n)))
    k = min(cap, int(n.value))
    return list(s[:k]), list(g[:k])


def release_workspace():
    _check(lib().emu_release_workspace())


def workspace_bytes() -> int:
    return int(lib().emu_workspace_bytes())
