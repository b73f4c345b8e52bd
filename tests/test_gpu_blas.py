"""GPU parity of the BLAS forms C = alpha op(A) op(B) + beta C (emu_sgemm_ex,
emu_dgemm_ex): transposed operands are packed from their stored layout and give
the bits of the plain call; the output update is fl(fl(alpha P) + fl(beta C))."""
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
    return E


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def stored(X, trans):
    return np.ascontiguousarray(X.T) if trans == "T" else X


CASES = [("N", "N"), ("T", "N"), ("N", "T"), ("T", "T")]
SHAPES = [(33, 17, 40), (130, 70, 600), (257, 129, 513)]


@pytest.mark.parametrize("ta,tb", CASES)
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("nprod", [6, 21])
def test_dgemm_ex_bit_exact(emu, ta, tb, shape, nprod):
    M, N, K = shape
    A = S.make("wide", 701, (M, K), np.float64)
    B = S.make("uniform", 702, (K, N), np.float64)
    C0 = S.make("normal", 703, (M, N), np.float64)
    for alpha, beta in ((1.0, 0.0), (-2.5, 0.75), (0.3, 0.0)):
        ref, _ = O.emu_dgemm_ex(stored(A, ta), stored(B, tb), nprod, C0, ta, tb, alpha, beta)
        got = emu.dgemm_ex(dev(stored(A, ta)), dev(stored(B, tb)), nprod, dev(C0.copy()), ta, tb,
                           alpha, beta).cpu().numpy()
        assert np.array_equal(got.view(np.uint64), ref.view(np.uint64)), (alpha, beta)


@pytest.mark.parametrize("ta,tb", CASES)
@pytest.mark.parametrize("shape", SHAPES)
def test_sgemm_ex_transposes_give_the_plain_bits(emu, ta, tb, shape):
    M, N, K = shape
    A = S.make("normal", 711, (M, K), np.float32)
    B = S.make("normal", 712, (K, N), np.float32)
    P = emu.sgemm(dev(A), dev(B)).cpu().numpy()
    got = emu.sgemm_ex(dev(stored(A, ta)), dev(stored(B, tb)), None, ta, tb).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), P.view(np.uint32))


@pytest.mark.parametrize("ta,tb", CASES)
@pytest.mark.parametrize("shape", SHAPES)
def test_sgemm_ex_against_the_oracle(emu, ta, tb, shape):
    """The SGEMM BLAS forms against the oracle's composition, at the bar of the
    plain emulated SGEMM: against the exact value alpha (AB) + beta C (FP64
    products of the FP32 inputs, double-double sums), the GPU's normwise error
    is at most twice the oracle's (plus the FP32 rounding of the update, which
    both pay), and each entry stays within the per-entry cap of the plain call
    scaled by |alpha|, plus one rounding of the output."""
    M, N, K = shape
    A = S.make("normal", 751, (M, K), np.float32)
    B = S.make("normal", 752, (K, N), np.float32)
    C0 = S.make("normal", 753, (M, N), np.float32)
    A64, B64 = A.astype(np.float64), B.astype(np.float64)
    hi, lo = O.ref_gemm_dd(A64, B64)
    absp = np.abs(A64) @ np.abs(B64)
    _, esc_cap = sgemm_bounds(K)
    for alpha, beta in ((1.0, 0.0), (-0.75, 0.5), (2.5, -1.25)):
        ref = (alpha * hi + beta * C0.astype(np.float64)) + alpha * lo
        orc, _ = O.emu_sgemm_ex(stored(A, ta), stored(B, tb), C0, ta, tb, alpha, beta)
        got = emu.sgemm_ex(dev(stored(A, ta)), dev(stored(B, tb)), dev(C0.copy()), ta, tb,
                           alpha, beta).cpu().numpy()
        e_gpu, e_orc = O.e_F(got, ref), O.e_F(orc, ref)
        assert e_gpu <= 2 * e_orc + 2.0 ** -24, (alpha, beta, e_gpu, e_orc)
        err = np.abs(got.astype(np.float64) - ref)
        cap = abs(alpha) * esc_cap * absp + 2.0 ** -23 * np.abs(ref)
        assert np.all(err <= cap), (alpha, beta, float(np.max(err / np.maximum(cap, 1e-300))))


def sgemm_bounds(K):
    """The absolute caps of the plain emulated SGEMM (normwise, per entry)."""
    return 4 * K * 2.0 ** -24, 2.0 ** -22 + (6 * 256 + -(-K // 256)) * 2.0 ** -24


@pytest.mark.parametrize("alpha,beta", [(2.0, 0.0), (-0.5, 1.0), (1.5, -3.25)])
def test_sgemm_ex_output_update_rounding(emu, alpha, beta):
    """The update on the GPU's own product P: fl(fl(alpha P) + fl(beta C))."""
    A = S.make("normal", 721, (150, 300), np.float32)
    B = S.make("normal", 722, (300, 90), np.float32)
    C0 = S.make("normal", 723, (150, 90), np.float32)
    P = emu.sgemm(dev(A), dev(B)).cpu().numpy()
    got = emu.sgemm_ex(dev(A), dev(B), dev(C0.copy()), "N", "N", alpha, beta).cpu().numpy()
    want = O._blas_out(P, C0, alpha, beta, np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_beta_zero_never_reads_c_and_alpha_zero_never_reads_ab(emu):
    A = S.make("normal", 731, (40, 50), np.float64)
    B = S.make("normal", 732, (50, 30), np.float64)
    Cnan = torch.full((40, 30), float("nan"), dtype=torch.float64, device="cuda")
    got = emu.dgemm_ex(dev(A), dev(B), 10, Cnan, "N", "N", 1.0, 0.0).cpu().numpy()
    ref, _ = O.emu_dgemm(A, B, 10)
    assert np.array_equal(got, ref)
    C0 = S.make("normal", 733, (40, 30), np.float64)
    Anan = torch.full((40, 50), float("nan"), dtype=torch.float64, device="cuda")
    got = emu.dgemm_ex(Anan, dev(B), 6, dev(C0.copy()), "N", "N", 0.0, -2.0).cpu().numpy()
    assert np.array_equal(got, -2.0 * C0)
    got = emu.sgemm_ex(Anan.float(), dev(B.astype(np.float32)), dev(C0.astype(np.float32)), "N",
                       "N", 0.0, 0.0).cpu().numpy()
    assert not got.any()


def test_dgemm_ex_rowcol_scope_with_transposes(emu):
    A = S.make("normal_scaled_rows", 741, (90, 200), np.float64)
    B = S.make("wide", 742, (200, 60), np.float64)
    C0 = S.make("normal", 743, (90, 60), np.float64)
    ref, _ = O.emu_dgemm_ex(A.T.copy(), B.T.copy(), 15, C0, "T", "T", 1.25, -1.0,
                            scope=O.SCOPE_ROWCOL)
    emu.set_split_scope(emu.SCOPE_ROWCOL)
    try:
        got = emu.dgemm_ex(dev(A.T), dev(B.T), 15, dev(C0.copy()), "T", "T", 1.25,
                           -1.0).cpu().numpy()
    finally:
        emu.set_split_scope(emu.SCOPE_OPERAND)
    assert np.array_equal(got, ref)
