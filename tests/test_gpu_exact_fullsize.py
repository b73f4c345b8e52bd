"""Exact parity of every output entry at the full workload sizes.

Integer operands make the emulated products exact, so the whole output can be
checked against the exact product instead of a sample:

  * DGEMM: integers |x| <= 2^15 split into two slices (A_0 a multiple of 2^7,
    A_1 the rest, |A_1| <= 2^6), so every product the split needs is retained
    from nprod = 6 on (Sec. 4.3; the integer pins of the oracle), and the
    reconstruction is the exact integer product AB.  Every partial sum is
    below 2^53, so the FP64 product of any BLAS is exact too;
  * SGEMM: BF16-exact integers |x| <= 16 (one component each, Sec. 4.2) whose
    every partial sum stays below 2^24, so FP32 accumulation in any order is
    exact.

At 8192 the exact product comes from the host's FP64 BLAS.  At
16384 x 16384 x 16384 the host would take minutes, so the exact product comes
from the device's native FP64 GEMM (torch.matmul, the vendor library: not this
library's path), itself checked against exact int64 dot products on two full
rows and two full columns.  The same 8192 launch is also compared with the
oracle along its whole first and last row on wide-range operands.
"""
import numpy as np
import pytest
import torch

import oracle as O
import seeded_inputs as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    yield E
    E.release_workspace()
    torch.cuda.empty_cache()


def ints(seed, shape, bound):
    """Seeded integers in [-bound, bound] (from the uniform[-1, 1] stream)."""
    return np.rint(S.make("uniform", seed, shape, np.float64) * bound)


def count_diff(got: np.ndarray, want: np.ndarray) -> int:
    return int(np.count_nonzero(got.view(np.uint64) != want.view(np.uint64)))


@pytest.fixture(scope="module")
def int8192():
    n = 8192
    A = ints(1201, (n, n), 2 ** 15)
    B = ints(1202, (n, n), 2 ** 15)
    return A, B, A @ B


@pytest.mark.parametrize("nprod", [6, 21])
def test_dgemm_8192_every_entry_exact(emu, int8192, nprod):
    A, B, exact = int8192
    print(f"dgemm 8192^3 integers nprod={nprod}", flush=True)
    C = emu.dgemm(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), nprod).cpu().numpy()
    assert count_diff(C, exact) == 0


def test_dgemm_16384_every_entry_exact(emu):
    n = 16384
    A = ints(1211, (n, n), 2 ** 15)
    B = ints(1212, (n, n), 2 ** 15)
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    print("native FP64 reference 16384^3 (vendor GEMM)", flush=True)
    ref = torch.matmul(dA, dB)
    torch.cuda.synchronize()
    # the reference is exact: check it against int64 dot products
    Ai, Bi = A.astype(np.int64), B.astype(np.int64)
    refh = ref.cpu().numpy()
    for r in (0, n - 1):
        assert np.array_equal(refh[r].astype(np.int64), Ai[r] @ Bi)
    for c in (0, n - 1):
        assert np.array_equal(refh[:, c].astype(np.int64), Ai @ Bi[:, c])
    del Ai, Bi
    for nprod in (6, 21):
        print(f"dgemm 16384^3 integers nprod={nprod}", flush=True)
        C = emu.dgemm(dA, dB, nprod)
        nd = int(torch.count_nonzero(C.view(torch.int64) != ref.view(torch.int64)).item())
        assert nd == 0, f"nprod={nprod}: {nd} entries differ from the exact product"
        del C
    del dA, dB, ref
    emu.release_workspace()
    torch.cuda.empty_cache()


def test_sgemm_8192_every_entry_exact(emu):
    n = 8192
    A = ints(1221, (n, n), 16).astype(np.float32)
    B = ints(1222, (n, n), 16).astype(np.float32)
    exact = A.astype(np.float64) @ B.astype(np.float64)
    assert np.max(np.abs(exact)) < 2 ** 24
    print("sgemm 8192^3 integers", flush=True)
    C = emu.sgemm(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()).cpu().numpy()
    assert np.array_equal(C.astype(np.float64), exact)


def test_dgemm_8192_first_and_last_row_against_the_oracle(emu):
    """Wide-range operands (config of the 8192 benchmark): rows 0 and M - 1,
    every column, bit-exact against the oracle."""
    n = 8192
    A = S.make("wide", 1231, (n, n), np.float64)
    B = S.make("wide", 1232, (n, n), np.float64)
    print("dgemm 8192^3 wide nprod=6 (rows 0 and M-1 vs oracle)", flush=True)
    C = emu.dgemm(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(), 6)
    rows = np.repeat(np.array([0, n - 1], np.int64), n)
    cols = np.tile(np.arange(n, dtype=np.int64), 2)
    got = C[torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()].cpu().numpy()
    del C
    ref, st = O.emu_dgemm_entries(A, B, rows, cols, 6)
    assert st == 0
    assert count_diff(got, ref) == 0
