"""GPU parity of the native FP64 fallback (emu_set_fallback(EMU_FALLBACK_FP64)).

Against the oracle's fallback form: in-domain calls keep the emulation's bits
and report no fallback; calls whose split raises a status bit give the plain
FP64 GEMM of the inputs, checked exactly where every product and partial sum
is an FP64 value, else within the FP64 GEMM bound 2 (K + 2) u (|alpha| |A||B| +
|beta| |C|) (u = 2^-53: both sides round each fused or separate multiply-add
once, in different orders), and report EMU_STATUS_FALLBACK.
"""
import ctypes
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as O
import seeded_inputs as S

pytestmark = pytest.mark.gpu
U = 2.0 ** -53


@pytest.fixture(scope="module")
def emu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    E.set_fallback(E.FALLBACK_FP64)
    yield E
    E.set_fallback(E.FALLBACK_NONE)
    E.set_split_scope(E.SCOPE_OPERAND)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def stored(X, trans):
    return np.ascontiguousarray(X.T) if trans == "T" else X


def out_of_domain(seed, M, N, K):
    """Integers |x| <= 100 with one entry of A below BF16's range that meets a
    row of B at 2^127: every exact output is an integer plus 0 or 3 2^-13."""
    rng = np.random.default_rng(seed)
    A = rng.integers(-100, 101, (M, K)).astype(np.float64)
    B = rng.integers(-100, 101, (K, N)).astype(np.float64)
    k = K // 2
    A[:, k] = 0.0
    A[M // 3, k] = 3.0 * 2.0 ** -140
    B[k, :] = 2.0 ** 127
    return A, B


@pytest.mark.parametrize("nprod", [6, 21])
def test_in_domain_keeps_the_emulation(emu, nprod):
    A = S.make("wide", 1301, (130, 700), np.float64)
    B = S.make("uniform", 1302, (700, 90), np.float64)
    emu.domain_status()
    got = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    assert emu.domain_status() == 0
    ref, st = O.emu_dgemm_ex(A, B, nprod, fallback=O.FALLBACK_FP64)
    assert st == 0 and np.array_equal(got.view(np.uint64), ref.view(np.uint64))


@pytest.mark.parametrize("shape", [(7, 5, 9), (130, 70, 600), (257, 129, 1500)])
def test_out_of_domain_gives_the_exact_product(emu, shape):
    M, N, K = shape
    A, B = out_of_domain(1303, M, N, K)
    emu.domain_status()
    got = emu.dgemm(dev(A), dev(B), 21).cpu().numpy()
    st = emu.domain_status()
    assert st & emu.STATUS_RANGE and st & emu.STATUS_FALLBACK
    ref, sto = O.emu_dgemm_ex(A, B, 21, fallback=O.FALLBACK_FP64)
    assert sto & O.ST_FALLBACK
    assert np.array_equal(got, ref)
    m = M // 3
    exact = sum(Fraction(float(A[m, k])) * Fraction(float(B[k, 0])) for k in range(K))
    assert Fraction(float(got[m, 0])) == exact


def test_infinities_follow_ieee(emu):
    A = S.make("normal", 1304, (40, 50), np.float64)
    B = S.make("normal", 1305, (50, 30), np.float64)
    A[3, 7] = np.inf
    B[11, 4] = -np.inf
    emu.domain_status()
    got = emu.dgemm(dev(A), dev(B), 10).cpu().numpy()
    st = emu.domain_status()
    assert st & emu.STATUS_NAN and st & emu.STATUS_FALLBACK
    want = A @ B
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(np.isinf(got), np.isinf(want))
    fin = np.isfinite(want)
    bound = 2 * 52 * U * (np.abs(A) @ np.abs(B))
    assert np.all(np.abs(got[fin] - want[fin]) <= bound[fin])


@pytest.mark.parametrize("ta,tb", [("N", "N"), ("T", "N"), ("N", "T"), ("T", "T")])
def test_blas_forms_with_beta(emu, ta, tb):
    """Out-of-domain wide-range inputs (one entry at 2^-150): alpha op(A) op(B)
    + beta C within the FP64 bound of the oracle's form; C is read as it was
    before the call."""
    M, N, K = 90, 70, 333
    A = S.make("wide", 1306, (M, K), np.float64)
    B = S.make("wide", 1307, (K, N), np.float64)
    A[5, 17] = 2.0 ** -150
    C0 = S.make("normal", 1308, (M, N), np.float64)
    alpha, beta = -1.25, 0.5
    got = emu.dgemm_ex(dev(stored(A, ta)), dev(stored(B, tb)), 15, dev(C0.copy()), ta, tb, alpha,
                       beta).cpu().numpy()
    assert emu.domain_status() & emu.STATUS_FALLBACK
    ref, st = O.emu_dgemm_ex(stored(A, ta), stored(B, tb), 15, C0, ta, tb, alpha, beta,
                             fallback=O.FALLBACK_FP64)
    assert st & O.ST_FALLBACK
    bound = 2 * (K + 2) * U * (abs(alpha) * (np.abs(A) @ np.abs(B)) + abs(beta) * np.abs(C0))
    assert np.all(np.abs(got - ref) <= bound)


def test_rowcol_scope_outside_its_domain(emu):
    """Entries more than 2^126 below their row's maximum leave the row/column
    scope's domain too: the fallback gives the exact product."""
    A, B = out_of_domain(1309, 64, 40, 300)
    A[:, 0] = 2.0 ** 20                     # each row's maximum far above 3 2^-140
    emu.set_split_scope(emu.SCOPE_ROWCOL)
    try:
        got = emu.dgemm(dev(A), dev(B), 21).cpu().numpy()
        st = emu.domain_status()
    finally:
        emu.set_split_scope(emu.SCOPE_OPERAND)
    assert st & emu.STATUS_FALLBACK
    ref, sto = O.emu_dgemm_ex(A, B, 21, scope=O.SCOPE_ROWCOL, fallback=O.FALLBACK_FP64)
    assert sto & O.ST_FALLBACK and np.array_equal(got, ref)


def test_noalloc_entry_point_falls_back_too(emu):
    A, B = out_of_domain(1310, 100, 60, 500)
    dA, dB = dev(A), dev(B)
    C = torch.empty((100, 60), dtype=torch.float64, device="cuda")
    L = emu.lib()
    L.emu_set_stream(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    emu.domain_status()
    assert L.emu_dgemm_noalloc(100, 60, 500, dA.data_ptr(), 500, dB.data_ptr(), 60, C.data_ptr(),
                               60, 21) == emu.EMU_OK
    assert emu.domain_status() & emu.STATUS_FALLBACK
    ref, _ = O.emu_dgemm_ex(A, B, 21, fallback=O.FALLBACK_FP64)
    assert np.array_equal(C.cpu().numpy(), ref)
