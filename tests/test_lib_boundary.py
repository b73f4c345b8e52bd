"""CPU-side checks of the C-ABI library (no kernel is launched).

The library must load, export every function include/emu.h declares, and
reject invalid arguments with EMU_EINVAL before touching the HIP runtime.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_04663_amd", "libemu.so")


def _declared():
    with open(os.path.join(ROOT, "include", "emu.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(emu_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LIB):
        pytest.fail("libemu.so is not built (run __graft_entry__.build())")
    import paper_2609_04663_amd as emu
    return emu.lib()


def test_header_declares_the_paper_entry_points():
    names = _declared()
    for n in ("emu_sgemm", "emu_dgemm", "emu_set_stream", "emu_domain_status",
              "emu_last_error", "emu_release_workspace", "emu_split_f32", "emu_split_f64"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    import paper_2609_04663_amd as emu
    for n in _declared():
        assert hasattr(L, n), n
    assert set(emu.EXPORTS) == set(_declared())


P = ctypes.c_void_p(0x1000)     # never dereferenced: validation fails first


@pytest.mark.parametrize("args", [
    (-1, 4, 4, P, 4, P, 4, P, 4),        # negative M
    (4, -1, 4, P, 4, P, 4, P, 4),        # negative N
    (4, 4, -1, P, 4, P, 4, P, 4),        # negative K
    (4, 4, 8, P, 7, P, 4, P, 4),         # lda < K
    (4, 8, 4, P, 4, P, 7, P, 8),         # ldb < N
    (4, 8, 4, P, 4, P, 8, P, 7),         # ldc < N
    (4, 4, 4, None, 4, P, 4, P, 4),      # NULL A
    (4, 4, 4, P, 4, None, 4, P, 4),      # NULL B
    (4, 4, 4, P, 4, P, 4, None, 4),      # NULL C
])
def test_gemm_invalid_arguments(L, args):
    import paper_2609_04663_amd as emu
    assert L.emu_sgemm(*args) == emu.EMU_EINVAL
    assert L.emu_last_error()
    assert L.emu_dgemm(*args, 10) == emu.EMU_EINVAL


@pytest.mark.parametrize("nprod", [0, 2, 4, 7, 20, 22, 34, 37, -6])
def test_dgemm_invalid_nprod(L, nprod):
    import paper_2609_04663_amd as emu
    assert L.emu_dgemm(4, 4, 4, P, 4, P, 4, P, 4, nprod) == emu.EMU_EINVAL


def test_dgemm_accepts_every_depth(L):
    """N_p(d) for d = 1 .. 11 pass validation (M = 0: no launch follows)."""
    import paper_2609_04663_amd as emu
    assert emu.NPROD_ALL == tuple(sum(1 for i in range(6) for j in range(6) if i + j < d)
                                  for d in range(1, 12))
    for nprod in emu.NPROD_ALL:
        assert L.emu_dgemm(0, 4, 4, P, 4, P, 4, P, 4, nprod) == emu.EMU_OK


def test_empty_output_is_a_no_op(L):
    import paper_2609_04663_amd as emu
    assert L.emu_sgemm(0, 4, 4, P, 4, P, 4, P, 4) == emu.EMU_OK
    assert L.emu_dgemm(4, 0, 4, P, 4, P, 1, P, 1, 6) == emu.EMU_OK


def test_split_hooks_invalid(L):
    import paper_2609_04663_amd as emu
    assert L.emu_split_f32(-1, 4, P, 4, 0, P) == emu.EMU_EINVAL
    assert L.emu_split_f32(4, 4, P, 3, 0, P) == emu.EMU_EINVAL
    assert L.emu_split_f32(4, 4, P, 4, 2, P) == emu.EMU_EINVAL
    assert L.emu_split_f64(4, 4, P, 4, 0, P, None) == emu.EMU_EINVAL


def test_split_mode_and_status_arguments(L):
    import paper_2609_04663_amd as emu
    assert L.emu_set_split_mode(2) == emu.EMU_EINVAL
    assert L.emu_set_split_mode(emu.SPLIT_LITERAL) == emu.EMU_OK
    assert L.emu_set_split_mode(emu.SPLIT_SYM) == emu.EMU_OK
    assert L.emu_domain_status(None) == emu.EMU_EINVAL
    assert L.emu_set_stream(None) == emu.EMU_OK


def test_split_scope_and_scale_hook_arguments(L):
    import paper_2609_04663_amd as emu
    assert L.emu_set_split_scope(3) == emu.EMU_EINVAL
    assert L.emu_set_split_scope(-1) == emu.EMU_EINVAL
    assert L.emu_set_split_scope(emu.SCOPE_KBIN) == emu.EMU_OK
    assert L.emu_set_split_scope(emu.SCOPE_ROWCOL) == emu.EMU_OK
    assert L.emu_set_split_scope(emu.SCOPE_OPERAND) == emu.EMU_OK
    assert L.emu_scale_exponents(-1, 4, P, 4, 0, P) == emu.EMU_EINVAL      # negative R
    assert L.emu_scale_exponents(4, 4, P, 3, 0, P) == emu.EMU_EINVAL       # ldx < Cc
    assert L.emu_scale_exponents(4, 4, P, 4, 2, P) == emu.EMU_EINVAL       # by_col
    assert L.emu_scale_exponents(4, 4, None, 4, 0, P) == emu.EMU_EINVAL    # NULL X
    assert L.emu_scale_exponents(4, 4, P, 4, 1, None) == emu.EMU_EINVAL    # NULL s
    assert L.emu_scale_exponents(0, 4, None, 4, 0, None) == emu.EMU_OK     # nothing to do


@pytest.mark.parametrize("ta,tb,args", [
    (b"X", b"N", (4, 4, 4, 1.0, P, 4, P, 4, 0.0, P, 4)),      # bad transa
    (b"N", b"Q", (4, 4, 4, 1.0, P, 4, P, 4, 0.0, P, 4)),      # bad transb
    (b"T", b"N", (8, 4, 4, 1.0, P, 4, P, 4, 0.0, P, 4)),      # A^T: lda < M
    (b"N", b"T", (4, 4, 8, 1.0, P, 8, P, 7, 0.0, P, 4)),      # B^T: ldb < K
    (b"N", b"N", (4, 8, 4, 1.0, P, 4, P, 8, 0.0, P, 7)),      # ldc < N
    (b"T", b"T", (-1, 4, 4, 1.0, P, 4, P, 4, 0.0, P, 4)),     # negative M
    (b"N", b"N", (4, 4, 4, 1.0, None, 4, P, 4, 0.0, P, 4)),   # NULL A with alpha != 0
])
def test_blas_forms_invalid_arguments(L, ta, tb, args):
    import paper_2609_04663_amd as emu
    assert L.emu_sgemm_ex(ta, tb, *args) == emu.EMU_EINVAL
    assert L.emu_dgemm_ex(ta, tb, *args, 6) == emu.EMU_EINVAL


def test_blas_forms_empty_output_and_nprod(L):
    import paper_2609_04663_amd as emu
    assert L.emu_sgemm_ex(b"T", b"T", 0, 4, 4, 1.0, P, 1, P, 4, 0.0, P, 4) == emu.EMU_OK
    assert L.emu_dgemm_ex(b"n", b"t", 4, 0, 4, 1.0, P, 4, P, 4, 0.0, P, 1, 21) == emu.EMU_OK
    assert L.emu_dgemm_ex(b"N", b"N", 4, 4, 4, 1.0, P, 4, P, 4, 0.0, P, 4, 7) == emu.EMU_EINVAL


@pytest.mark.parametrize("cshape", [(1, 6), (4, 6), (5, 5), (5, 7), (6, 6)])
def test_binding_rejects_wrong_output_shape(cshape):
    """A caller-supplied C must be M x N: the library writes M rows of ldc
    entries and a smaller C would be overrun.  The binding checks shapes from
    tensor metadata before any device work, so host tensors reach the check."""
    import torch
    import paper_2609_04663_amd as emu
    M, N, K = 5, 6, 3
    for dt, fn, extra in ((torch.float32, emu.sgemm, ()), (torch.float64, emu.dgemm, (6,))):
        A = torch.zeros((M, K), dtype=dt)
        B = torch.zeros((K, N), dtype=dt)
        C = torch.zeros(cshape, dtype=dt)
        with pytest.raises(ValueError, match="C must be"):
            fn(A, B, *extra, C=C)
    for dt, fn, extra in ((torch.float32, emu.sgemm_ex, ()), (torch.float64, emu.dgemm_ex, (6,))):
        A = torch.zeros((K, M), dtype=dt)                 # stored transposed
        B = torch.zeros((N, K), dtype=dt)
        C = torch.zeros(cshape, dtype=dt)
        with pytest.raises(ValueError, match="C must be"):
            fn(A, B, *extra, C=C, transa="T", transb="T")


def test_binding_needs_gpu_tensors_after_the_shape_checks():
    import torch
    import paper_2609_04663_amd as emu
    A = torch.zeros((5, 3), dtype=torch.float64)
    B = torch.zeros((3, 6), dtype=torch.float64)
    with pytest.raises(TypeError, match="GPU tensor"):
        emu.dgemm(A, B, 6, C=torch.zeros((5, 6), dtype=torch.float64))


def test_mode_switch_arguments(L):
    import paper_2609_04663_amd as emu
    for bad in (-1, 2):
        assert L.emu_set_sgemm_split(bad) == emu.EMU_EINVAL
        assert L.emu_set_fallback(bad) == emu.EMU_EINVAL
    for mode in (emu.SGEMM_SPLIT_STREAMED, emu.SGEMM_SPLIT_PASS):
        assert L.emu_set_sgemm_split(mode) == emu.EMU_OK
    for mode in (emu.FALLBACK_FP64, emu.FALLBACK_NONE):
        assert L.emu_set_fallback(mode) == emu.EMU_OK
