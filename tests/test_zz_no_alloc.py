"""The allocation-free entry point emu_dgemm_noalloc against emu_dgemm.

Called through the C ABI (ctypes) with torch-owned device buffers: the result
must be bit-identical to emu_dgemm's on the same inputs, on consecutive calls
that share the fixed scratch (the second one smaller, so stale planes of the
first call sit beyond what it reads), without the library's workspace ever
being allocated; sizes beyond the scratch are refused before any launch, and
the status word of the scratch reaches emu_domain_status.
"""
import ctypes

import numpy as np
import pytest
import torch

import seeded_inputs as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    return E


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def noalloc(emu, A, B, C, nprod):
    """emu_dgemm_noalloc through the C ABI on the current stream."""
    L = emu.lib()
    M, K = A.shape
    N = B.shape[1]
    L.emu_set_stream(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return L.emu_dgemm_noalloc(M, N, K, A.data_ptr(), A.stride(0), B.data_ptr(), B.stride(0),
                               C.data_ptr(), C.stride(0), nprod)


@pytest.mark.parametrize("nprod", [6, 21])
def test_noalloc_matches_dgemm_on_consecutive_calls(emu, nprod):
    emu.release_workspace()
    shapes = [(700, 650, 900), (130, 70, 300)]          # the second call is smaller
    outs = []
    for i, (M, N, K) in enumerate(shapes):
        A = dev(S.make("wide", 901 + 2 * i, (M, K), np.float64))
        B = dev(S.make("uniform", 902 + 2 * i, (K, N), np.float64))
        C = torch.full((M, N), float("nan"), dtype=torch.float64, device="cuda")
        assert noalloc(emu, A, B, C, nprod) == emu.EMU_OK, emu.lib().emu_last_error()
        torch.cuda.synchronize()
        assert emu.workspace_bytes() == 0                # nothing was allocated
        outs.append((A, B, C.cpu().numpy()))
    assert emu.domain_status() == 0
    for A, B, got in outs:
        ref = emu.dgemm(A, B, nprod).cpu().numpy()
        assert np.array_equal(got.view(np.uint64), ref.view(np.uint64))


def test_noalloc_padded_leading_dimensions(emu):
    M, N, K = 257, 129, 513
    A = dev(np.pad(S.make("wide", 911, (M, K), np.float64), ((0, 0), (0, 7))))[:, :K]
    B = dev(np.pad(S.make("wide", 912, (K, N), np.float64), ((0, 0), (0, 3))))[:, :N]
    C = torch.zeros((M, N + 5), dtype=torch.float64, device="cuda")
    assert noalloc(emu, A, B, C[:, :N], 15) == emu.EMU_OK
    ref = emu.dgemm(A, B, 15).cpu().numpy()
    assert np.array_equal(C[:, :N].cpu().numpy(), ref)
    assert not C[:, N:].cpu().numpy().any()              # nothing written past N


def test_noalloc_refuses_sizes_beyond_the_scratch(emu):
    L = emu.lib()
    P = ctypes.c_void_p(0x1000)                          # never dereferenced
    assert L.emu_dgemm_noalloc(4096, 4096, 4096, P, 4096, P, 4096, P, 4096, 21) == emu.EMU_ENOMEM
    assert b"scratch" in L.emu_last_error()
    assert L.emu_dgemm_noalloc(4, 4, 4, P, 4, P, 4, P, 4, 7) == emu.EMU_EINVAL


def test_noalloc_reports_status(emu):
    A = dev(np.ldexp(S.make("uniform", 921, (60, 300), np.float64), -45))
    B = dev(np.ldexp(S.make("uniform", 922, (300, 40), np.float64), -45))
    C = torch.empty((60, 40), dtype=torch.float64, device="cuda")
    emu.domain_status()
    assert noalloc(emu, A, B, C, 21) == emu.EMU_OK
    assert emu.domain_status() == emu.STATUS_INEXACT
    assert noalloc(emu, A, B, C, 6) == emu.EMU_OK
    assert emu.domain_status() == 0
