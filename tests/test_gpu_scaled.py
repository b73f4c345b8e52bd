"""GPU parity of the scale-aware FP64 split (row weights of A, column weights of
B, EMU_SCOPE_ROWCOL) against the oracle's form of it: weights, split and DGEMM
bit-exact, the widened domain, and the full-size rectangular workload."""
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


@pytest.fixture
def rowcol(emu):
    emu.set_split_scope(emu.SCOPE_ROWCOL)
    yield emu
    emu.set_split_scope(emu.SCOPE_OPERAND)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def padded_view(a, extra=3):
    R, C = a.shape
    big = np.zeros((R, C + extra), dtype=a.dtype)
    big[:, :C] = a
    return dev(big)[:, :C]


def special_matrix():
    X = S.make("wide", 601, (70, 130), np.float64)
    X[3] = 0.0                                  # empty row
    X[:, 5] = 0.0                               # empty column
    X[7] *= 2.0 ** 300                          # far outside the BF16 range
    X[9] *= 2.0 ** -400
    X[11, 17] = np.inf                          # ignored by the weights
    X[:, 20] *= 2.0 ** -200
    return X


@pytest.mark.parametrize("by_col", [0, 1])
def test_scale_exponents_bit_exact(emu, by_col):
    X = special_matrix()
    got = emu.scale_exponents(padded_view(X), by_col=bool(by_col)).cpu().numpy()
    assert np.array_equal(got, O.scale_exponents(X, by_col=bool(by_col)))


@pytest.mark.parametrize("as_b", [0, 1])
@pytest.mark.parametrize("dist", ["uniform", "normal_scaled_rows", "wide"])
def test_split_f64_rowcol_bit_exact(rowcol, as_b, dist):
    X = S.make(dist, 611, (90, 140), np.float64)
    s = O.scale_exponents(X, by_col=bool(as_b))
    Xs = np.ldexp(X, -(s[None, :] if as_b else s[:, None]))
    ref, vref, _, _ = O.split_f64(Xs)
    slices, v = rowcol.split_f64(padded_view(X), as_b=bool(as_b))
    assert np.array_equal(slices.cpu().numpy().view(np.uint16), ref)
    assert np.array_equal(v.cpu().numpy(), vref)


GEMM_SHAPES = [(1, 1, 1), (33, 17, 40), (130, 70, 600), (257, 129, 513)]


@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
@pytest.mark.parametrize("dist", ["normal_scaled_rows", "wide"])
def test_dgemm_rowcol_bit_exact(rowcol, shape, nprod, dist):
    M, N, K = shape
    A = S.make(dist, 621, (M, K), np.float64)
    B = S.make(dist, 622, (K, N), np.float64)
    ref, st = O.emu_dgemm(A, B, nprod, scope=O.SCOPE_ROWCOL)
    rowcol.domain_status()
    C = rowcol.dgemm(padded_view(A), padded_view(B), nprod).cpu().numpy()
    assert rowcol.domain_status() == st
    assert np.array_equal(C.view(np.uint64), ref.view(np.uint64)), \
        f"{np.count_nonzero(C != ref)} of {C.size} differ"


def test_dgemm_rowcol_beyond_bf16_range(rowcol):
    """Rows near 1e200 and columns near 1e-200: out of the paper's domain,
    in range with weights; bit-exact with the oracle and FP64-accurate."""
    A = S.make("uniform", 631, (100, 300), np.float64) * 1e200
    B = S.make("uniform", 632, (300, 80), np.float64) * 1e-200
    A[::7] *= 1e-150
    ref, st = O.emu_dgemm(A, B, 21, scope=O.SCOPE_ROWCOL)
    assert st == 0
    rowcol.domain_status()
    C = rowcol.dgemm(dev(A), dev(B), 21).cpu().numpy()
    assert rowcol.domain_status() == 0
    assert np.array_equal(C, ref)
    hi, _ = O.ref_gemm_dd(A, B)
    assert O.e_F(C, hi) < 4e-16


def test_operand_scope_flags_what_rowcol_accepts(emu):
    A = S.make("uniform", 641, (40, 64), np.float64) * 1e200
    B = S.make("uniform", 642, (64, 40), np.float64)
    emu.set_split_scope(emu.SCOPE_OPERAND)
    emu.domain_status()
    emu.dgemm(dev(A), dev(B), 6)
    assert emu.domain_status() & emu.STATUS_RANGE


@pytest.mark.parametrize("shape", [(16384, 16384, 512), (1024, 1024, 65536)])
def test_rectangular_scaled_rows_rowcol(rowcol, shape):
    """The rectangular workloads with 1 % of the rows scaled by 2^16, nprod 10,
    in the ROWCOL scope: sampled entries bit-exact, and the error on the A rows
    that were not scaled drops well below the operand-wide split's."""
    M, N, K = shape
    sa, sb = S.seeds(5)
    A = S.make("normal_scaled_rows", sa, (M, K), np.float64)
    B = S.make("normal_scaled_rows", sb, (K, N), np.float64)
    rng = np.random.default_rng(M + K)
    big = np.abs(A).max(axis=1) > 2.0 ** 10
    rows = rng.choice(np.flatnonzero(~big), 192)
    cols = rng.integers(0, N, 192)
    dA, dB = dev(A), dev(B)
    r_t, c_t = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    C = rowcol.dgemm(dA, dB, 10)
    got = C[r_t, c_t].cpu().numpy()
    del C
    ref, st = O.emu_dgemm_entries(A, B, rows, cols, 10, scope=O.SCOPE_ROWCOL)
    assert np.array_equal(got, ref)
    rowcol.set_split_scope(rowcol.SCOPE_OPERAND)
    C = rowcol.dgemm(dA, dB, 10)
    got_op = C[r_t, c_t].cpu().numpy()
    del C, dA, dB
    hi, _ = O.ref_dd_entries(A, B, rows, cols)
    e_rc, e_op = O.e_F(got, hi), O.e_F(got_op, hi)
    print(f"{shape}: unscaled-row e_F rowcol {e_rc:.3e} operand-wide {e_op:.3e}", flush=True)
    assert e_rc < e_op / 10
    rowcol.release_workspace()
    torch.cuda.empty_cache()
