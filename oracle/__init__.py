"""CPU oracle for BF16 component-product emulation of FP32/FP64 GEMM (arxiv 2609.04663).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP implementation in ``paper_2609_04663_amd``: the arithmetic lives in
``oracle.c`` (plain C, FP64 where the paper does not fix the precision), and this
module only marshals numpy arrays through ctypes and evaluates the paper's
accuracy metrics.

Functions (all operands row-major numpy arrays, all on the host):

* ``split_f32(X)``       -> uint16 [3, R, C]     Eq. (fp32split), Sec. 4.2
* ``split_f64(X, mode)`` -> (uint16 [6, R, C], v[6], residual A^(6), status)
                                                  Eq. (fp64split), Sec. 4.3
* ``emu_sgemm(A, B)``    -> FP32 C               Algorithm fp32 + Sec. 6.2/6.3 order
* ``emu_dgemm(A, B, nprod, mode, scope)`` -> FP64 C   Algorithm fp64, Eq. (fp64reconstruction)
* ``scale_exponents(X, by_col)`` -> per-row / per-column power-of-two weights of
                                    the scale-aware split (Eq. ozakiscaled, Sec. 9)
* ``*_entries``          -> the same for selected (row, col) entries
* ``ref_gemm_f64``, ``ref_gemm_dd``, ``ref_dd_entries`` -> references
* ``e_F``, ``e_scaled``  -> Eq. (froerror) and Eq. (scalederror), Sec. 7.3
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

SPLIT_SYM = 0
SPLIT_LITERAL = 1
# Exponent scope of the FP64 split: the paper's operand-wide maxima (default),
# or the scale-aware form named as future work in Sec. 9: every row of A and
# every column of B is first divided by a stored power-of-two weight 2^s with
# s = ceil(log2 max|row|) (the per-row form of the weights 2^v of
# Eq. ozakiscaled), split operand-wide, and the weights are multiplied back
# into the FP64 result, C_mn = 2^(sA_m + sB_n) C'_mn.
SCOPE_OPERAND = 0
SCOPE_ROWCOL = 1
# K-binned scope (an extension of the scale-aware split along the reduction):
# the reduction indices k are grouped by the magnitude class of their product
# terms, every group is computed as its own row/column-scaled emulated GEMM
# (its own weights and exponent chains) and the groups are added in FP64,
# group 0 (the largest terms) first.  The class of k is
#   floor(-(ceil(log2 max_m |A~_mk|) + ceil(log2 max_n |B~_kn|)) / KBIN_WIDTH),
# capped at KBIN_MAX - 1, with A~, B~ the row- and column-scaled operands of
# the ROWCOL scope; a k whose column of A~ or row of B~ is zero contributes
# exact zeros and is left out.
SCOPE_KBIN = 2
KBIN_WIDTH = 8
KBIN_MAX = 8
# Fallback (the "fallback handling" of Sec. 9 for inputs the split cannot
# represent): when a DGEMM's status has any bit set, its product is the plain
# FP64 GEMM of the inputs instead, and status bit ST_FALLBACK is added.
FALLBACK_NONE = 0
FALLBACK_FP64 = 1
KC = 256  # reduction-panel length B_K of the paper's blocked loop (Sec. 6.1)

ST_NAN, ST_RANGE, ST_SUBNORMAL, ST_OVERFLOW, ST_INEXACT32, ST_FALLBACK = 1, 2, 4, 8, 16, 32
# N_p(d) = |S_d| of Eq. (product-selection), six slices per operand, d = 1 .. 11
NPROD_TO_D = {sum(1 for i in range(6) for j in range(6) if i + j < d): d for d in range(1, 12)}


def compile_source(src: str, out: str) -> str:
    """Compile a C source file into the shared library ``out`` with the oracle's
    flags (no fast-math, no FMA contraction)."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
           "-Wall", "-shared", "-fPIC", src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_source(_SRC, _LIB)
    return _LIB


_lib = None


@contextlib.contextmanager
def using_library(path: str):
    """Route every call of this module through another build of the oracle
    (the mutation tests use it to show that the pins reject planted mistakes)."""
    global _lib
    saved = _lib
    _lib = _configure(ctypes.CDLL(os.path.abspath(path)))
    try:
        yield
    finally:
        _lib = saved


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = _configure(ctypes.CDLL(_LIB))
    return _lib


def _configure(L):
    """Declare the argument and result types of the oracle's C functions."""
    i64, p, u32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_uint32
    L.orc_bf16_rne_f32.argtypes = [ctypes.c_float]
    L.orc_bf16_rne_f32.restype = ctypes.c_uint16
    L.orc_bf16_rne_f64.argtypes = [ctypes.c_double]
    L.orc_bf16_rne_f64.restype = ctypes.c_uint16
    L.orc_split_f32.argtypes = [i64, i64, p, i64, p]
    L.orc_split_f32.restype = u32
    L.orc_split_f64.argtypes = [i64, i64, p, i64, ctypes.c_int, p, p, p]
    L.orc_split_f64.restype = u32
    L.orc_emu_sgemm.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, i64]
    L.orc_emu_sgemm.restype = u32
    L.orc_emu_sgemm_entries.argtypes = [i64, i64, i64, p, i64, p, i64, i64, p, p, p, i64]
    L.orc_emu_sgemm_entries.restype = u32
    L.orc_emu_dgemm.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, ctypes.c_int,
                                ctypes.c_int, i64]
    L.orc_emu_dgemm.restype = u32
    L.orc_emu_dgemm_entries.argtypes = [i64, i64, i64, p, i64, p, i64, i64, p, p, p,
                                        ctypes.c_int, ctypes.c_int, i64]
    L.orc_emu_dgemm_entries.restype = u32
    L.orc_ref_gemm_f64.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64]
    L.orc_ref_gemm_dd.argtypes = [i64, i64, i64, p, i64, p, i64, p, p, i64]
    L.orc_ref_dd_entries.argtypes = [i64, i64, i64, p, i64, p, i64, i64, p, p, p, p]
    L.orc_absprod_entries.argtypes = [i64, p, i64, p, i64, i64, p, p, p]
    L.orc_num_threads.restype = ctypes.c_int
    L.orc_set_num_threads.argtypes = [ctypes.c_int]
    L.orc_sgemm_entries_from_comps.argtypes = [i64, i64, i64, p, p, i64, p, p, p, i64]
    L.orc_dgemm_entries_from_slices.argtypes = [i64, i64, i64, p, p, i64, p, p, p, ctypes.c_int,
                                                i64]
    L.orc_dgemm_entries_from_slices.restype = u32
    L.orc_dot_bf16_f32.argtypes = [i64, p, p]
    L.orc_dot_bf16_f32.restype = ctypes.c_float
    return L


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.asarray(a)
    assert a.dtype == dtype, f"expected {dtype}, got {a.dtype}"
    return np.ascontiguousarray(a)


def num_threads() -> int:
    return lib().orc_num_threads()


def set_num_threads(n: int):
    """Threads of the oracle's OpenMP loops from now on."""
    lib().orc_set_num_threads(int(n))


def sgemm_entries_from_comps(Av, Bv, rows, cols, kc: int = KC):
    """Entries (rows[e], cols[e]) of the emulated SGEMM from the components of
    split_f32 (Av [3, M, K], Bv [3, K, N])."""
    Av, Bv = _c(Av, np.uint16), _c(Bv, np.uint16)
    _, M, K = Av.shape
    N = Bv.shape[2]
    r, c = _idx(rows, cols)
    out = np.zeros(r.shape, dtype=np.float32)
    lib().orc_sgemm_entries_from_comps(M, N, K, _ptr(Av), _ptr(Bv), r.size, _ptr(r), _ptr(c),
                                       _ptr(out), int(kc))
    return out


def dgemm_entries_from_slices(Av, Bv, rows, cols, nprod: int, kc: int = KC):
    """Entries of the emulated DGEMM from the slices of split_f64 (Av [6, M, K],
    Bv [6, K, N]); returns (values, inexact-panel status)."""
    Av, Bv = _c(Av, np.uint16), _c(Bv, np.uint16)
    _, M, K = Av.shape
    N = Bv.shape[2]
    r, c = _idx(rows, cols)
    out = np.zeros(r.shape, dtype=np.float64)
    st = lib().orc_dgemm_entries_from_slices(M, N, K, _ptr(Av), _ptr(Bv), r.size, _ptr(r),
                                             _ptr(c), _ptr(out), int(nprod), int(kc))
    return out, int(st)


def bf16_rne_f32(x: float) -> int:
    return int(lib().orc_bf16_rne_f32(float(x)))


def bf16_rne_f64(x: float) -> int:
    return int(lib().orc_bf16_rne_f64(float(x)))


def dot_bf16_f32(x_bits: np.ndarray, y_bits: np.ndarray) -> float:
    """fl_32 of the exact dot product of two BF16 vectors (bit patterns)."""
    x = np.ascontiguousarray(np.asarray(x_bits, dtype=np.uint16))
    y = np.ascontiguousarray(np.asarray(y_bits, dtype=np.uint16))
    assert x.shape == y.shape
    return float(lib().orc_dot_bf16_f32(x.size, _ptr(x), _ptr(y)))


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    """Exact value of BF16 bit patterns (upper half of binary32)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def split_f32(X: np.ndarray):
    X = _c(X, np.float32)
    R, C = X.shape
    out = np.zeros((3, R, C), dtype=np.uint16)
    st = lib().orc_split_f32(R, C, _ptr(X), C, _ptr(out))
    return out, int(st)


def split_f64(X: np.ndarray, mode: int = SPLIT_SYM):
    X = _c(X, np.float64)
    R, C = X.shape
    out = np.zeros((6, R, C), dtype=np.uint16)
    v = np.zeros(6, dtype=np.int32)
    res = np.zeros((R, C), dtype=np.float64)
    st = lib().orc_split_f64(R, C, _ptr(X), C, int(mode), _ptr(out), _ptr(v), _ptr(res))
    return out, v, res, int(st)


def emu_sgemm(A: np.ndarray, B: np.ndarray, kc: int = KC):
    A, B = _c(A, np.float32), _c(B, np.float32)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.zeros((M, N), dtype=np.float32)
    st = lib().orc_emu_sgemm(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(C), N, int(kc))
    return C, int(st)


def _idx(rows, cols):
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    c = np.ascontiguousarray(np.asarray(cols, dtype=np.int64))
    assert r.shape == c.shape
    return r, c


def emu_sgemm_entries(A, B, rows, cols, kc: int = KC):
    A, B = _c(A, np.float32), _c(B, np.float32)
    M, K = A.shape
    N = B.shape[1]
    r, c = _idx(rows, cols)
    out = np.zeros(r.shape, dtype=np.float32)
    st = lib().orc_emu_sgemm_entries(M, N, K, _ptr(A), K, _ptr(B), N, r.size, _ptr(r), _ptr(c),
                                     _ptr(out), int(kc))
    return out, int(st)


def scale_exponents(X: np.ndarray, by_col: bool = False) -> np.ndarray:
    """ceil(log2 max|x|) over each row (or column) of X, from the exact
    frexp decomposition; 0 for a row without nonzero finite entries."""
    X = np.asarray(X, dtype=np.float64)
    a = np.where(np.isfinite(X), np.abs(X), 0.0)
    m = a.max(axis=0 if by_col else 1) if X.size else np.zeros(X.shape[1 if by_col else 0])
    f, e = np.frexp(m)
    s = np.where(f == 0.5, e - 1, e)
    return np.where(m > 0, s, 0).astype(np.int32)


def scaled_operands(A: np.ndarray, B: np.ndarray):
    """(sA, sB, A 2^-sA by rows, B 2^-sB by columns): exact power-of-two scalings."""
    sA = scale_exponents(A, by_col=False)
    sB = scale_exponents(B, by_col=True)
    return sA, sB, np.ldexp(A, -sA[:, None]), np.ldexp(B, -sB[None, :])


def _ceil_log2_or_none(m: np.ndarray):
    f, e = np.frexp(m)
    return np.where(f == 0.5, e - 1, e)


def kbin_classes(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Class of every reduction index k of the K-binned scope (-1: left out)."""
    _, _, As, Bs = scaled_operands(A, B)
    a = np.where(np.isfinite(As), np.abs(As), 0.0).max(axis=0) if As.shape[0] else np.zeros(As.shape[1])
    b = np.where(np.isfinite(Bs), np.abs(Bs), 0.0).max(axis=1) if Bs.shape[1] else np.zeros(Bs.shape[0])
    e = _ceil_log2_or_none(a) + _ceil_log2_or_none(b)
    cls = np.minimum((-e) // KBIN_WIDTH, KBIN_MAX - 1)
    return np.where((a > 0) & (b > 0), cls, -1).astype(np.int64)


def emu_dgemm(A: np.ndarray, B: np.ndarray, nprod: int, mode: int = SPLIT_SYM, kc: int = KC,
              scope: int = SCOPE_OPERAND):
    if scope == SCOPE_KBIN:
        A, B = _c(A, np.float64), _c(B, np.float64)
        cls = kbin_classes(A, B)
        C = np.zeros((A.shape[0], B.shape[1]), dtype=np.float64)
        st = 0
        first = True
        for b in range(KBIN_MAX):
            ks = np.nonzero(cls == b)[0]
            if ks.size == 0:
                continue
            Cb, sb = emu_dgemm(np.ascontiguousarray(A[:, ks]), np.ascontiguousarray(B[ks, :]),
                               nprod, mode, kc, SCOPE_ROWCOL)
            C = Cb if first else Cb + C            # FP64, group order
            first = False
            st |= sb
        return C, st
    if scope == SCOPE_ROWCOL:
        sA, sB, As, Bs = scaled_operands(_c(A, np.float64), _c(B, np.float64))
        C, st = emu_dgemm(As, Bs, nprod, mode, kc)
        return np.ldexp(C, sA[:, None] + sB[None, :]), st
    A, B = _c(A, np.float64), _c(B, np.float64)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2 and nprod in NPROD_TO_D
    C = np.zeros((M, N), dtype=np.float64)
    st = lib().orc_emu_dgemm(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(C), N, int(nprod), int(mode),
                             int(kc))
    return C, int(st)


def emu_dgemm_entries(A, B, rows, cols, nprod: int, mode: int = SPLIT_SYM, kc: int = KC,
                      scope: int = SCOPE_OPERAND):
    if scope == SCOPE_KBIN:
        A, B = _c(A, np.float64), _c(B, np.float64)
        cls = kbin_classes(A, B)
        r, c = _idx(rows, cols)
        out = np.zeros(r.shape, dtype=np.float64)
        st = 0
        first = True
        for b in range(KBIN_MAX):
            ks = np.nonzero(cls == b)[0]
            if ks.size == 0:
                continue
            ob, sb = emu_dgemm_entries(np.ascontiguousarray(A[:, ks]),
                                       np.ascontiguousarray(B[ks, :]), r, c, nprod, mode, kc,
                                       SCOPE_ROWCOL)
            out = ob if first else ob + out
            first = False
            st |= sb
        return out, st
    if scope == SCOPE_ROWCOL:
        sA, sB, As, Bs = scaled_operands(_c(A, np.float64), _c(B, np.float64))
        r, c = _idx(rows, cols)
        out, st = emu_dgemm_entries(As, Bs, r, c, nprod, mode, kc)
        return np.ldexp(out, sA[r] + sB[c]), st
    A, B = _c(A, np.float64), _c(B, np.float64)
    M, K = A.shape
    N = B.shape[1]
    r, c = _idx(rows, cols)
    out = np.zeros(r.shape, dtype=np.float64)
    st = lib().orc_emu_dgemm_entries(M, N, K, _ptr(A), K, _ptr(B), N, r.size, _ptr(r), _ptr(c),
                                     _ptr(out), int(nprod), int(mode), int(kc))
    return out, int(st)


def _blas_out(P, C, alpha, beta, dtype):
    """fl(alpha P) when beta == 0 (C unread), else fl(fl(alpha P) + fl(beta C)),
    in the output precision, elementwise (numpy rounds every operation)."""
    a, b = dtype(alpha), dtype(beta)
    if b == 0:
        return (a * P).astype(dtype)
    return (a * P + b * np.asarray(C, dtype=dtype)).astype(dtype)


def _scale_only(C, beta, shape, dtype):
    """The alpha == 0 or K == 0 result: beta C, or 0 when beta == 0 (C unread)."""
    b = dtype(beta)
    return np.zeros(shape, dtype) if b == 0 else (b * np.asarray(C, dtype=dtype)).astype(dtype)


def _op(X, trans):
    return np.ascontiguousarray(X.T) if trans in ("T", "t", "C", "c") else X


def emu_sgemm_ex(A, B, C=None, transa="N", transb="N", alpha=1.0, beta=0.0, kc: int = KC):
    """The BLAS form alpha op(A) op(B) + beta C (row-major, A and B as stored)."""
    opA, opB = _op(_c(A, np.float32), transa), _op(_c(B, np.float32), transb)
    M, N = opA.shape[0], opB.shape[1]
    if alpha == 0 or opA.shape[1] == 0:
        return _scale_only(C, beta, (M, N), np.float32), 0
    P, st = emu_sgemm(opA, opB, kc)
    return _blas_out(P, C, alpha, beta, np.float32), st


def emu_dgemm_ex(A, B, nprod: int, C=None, transa="N", transb="N", alpha=1.0, beta=0.0,
                 mode: int = SPLIT_SYM, kc: int = KC, scope: int = SCOPE_OPERAND,
                 fallback: int = FALLBACK_NONE):
    opA, opB = _op(_c(A, np.float64), transa), _op(_c(B, np.float64), transb)
    M, N = opA.shape[0], opB.shape[1]
    if alpha == 0 or opA.shape[1] == 0:
        return _scale_only(C, beta, (M, N), np.float64), 0
    P, st = emu_dgemm(opA, opB, nprod, mode, kc, scope)
    if fallback == FALLBACK_FP64 and st != 0:
        P = ref_gemm_f64(opA, opB)                 # the plain FP64 GEMM of the inputs
        st |= ST_FALLBACK
    return _blas_out(P, C, alpha, beta, np.float64), st


def ref_gemm_f64(A, B):
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float64))
    M, K = A.shape
    N = B.shape[1]
    C = np.zeros((M, N), dtype=np.float64)
    lib().orc_ref_gemm_f64(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(C), N)
    return C


def ref_gemm_dd(A, B):
    """Double-double reference: returns (hi, lo) with C ~ hi + lo."""
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float64))
    M, K = A.shape
    N = B.shape[1]
    hi = np.zeros((M, N), dtype=np.float64)
    lo = np.zeros((M, N), dtype=np.float64)
    lib().orc_ref_gemm_dd(M, N, K, _ptr(A), K, _ptr(B), N, _ptr(hi), _ptr(lo), N)
    return hi, lo


def ref_dd_entries(A, B, rows, cols):
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float64))
    M, K = A.shape
    N = B.shape[1]
    r, c = _idx(rows, cols)
    hi = np.zeros(r.shape, dtype=np.float64)
    lo = np.zeros(r.shape, dtype=np.float64)
    lib().orc_ref_dd_entries(M, N, K, _ptr(A), K, _ptr(B), N, r.size, _ptr(r), _ptr(c),
                             _ptr(hi), _ptr(lo))
    return hi, lo


def absprod_entries(A, B, rows, cols):
    """(|A||B|)_ij in FP64 for the selected entries (scaled-error denominator)."""
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64))
    B = np.ascontiguousarray(np.asarray(B, dtype=np.float64))
    K = A.shape[1]
    N = B.shape[1]
    r, c = _idx(rows, cols)
    out = np.zeros(r.shape, dtype=np.float64)
    lib().orc_absprod_entries(K, _ptr(A), K, _ptr(B), N, r.size, _ptr(r), _ptr(c), _ptr(out))
    return out


# ---------------------------------------------------------------------------
# Accuracy metrics, Sec. 7.3.

def _diff(Chat, ref):
    """Chat - ref, with ref either an array or a (hi, lo) double-double pair."""
    Chat = np.asarray(Chat, dtype=np.float64)
    if isinstance(ref, tuple):
        hi, lo = ref
        return (Chat - hi) - lo, hi + lo
    ref = np.asarray(ref, dtype=np.float64)
    return Chat - ref, ref


def e_F(Chat, ref) -> float:
    """Frobenius-norm relative error, Eq. (froerror)."""
    d, r = _diff(Chat, ref)
    den = float(np.linalg.norm(r.ravel()))
    return float(np.linalg.norm(d.ravel())) / den if den > 0 else float("nan")


def e_scaled(Chat, ref, absprod):
    """GEMM-scaled componentwise error, Eq. (scalederror).

    Returns (max over entries with a nonzero denominator, max absolute error over
    entries whose denominator is zero) -- the latter reported separately."""
    d, _ = _diff(Chat, ref)
    den = np.asarray(absprod, dtype=np.float64)
    nz = den > 0
    scaled = float(np.max(np.abs(d[nz]) / den[nz])) if nz.any() else 0.0
    zero_abs = float(np.max(np.abs(d[~nz]))) if (~nz).any() else 0.0
    return scaled, zero_abs
