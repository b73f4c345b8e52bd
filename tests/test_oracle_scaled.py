"""Scale-aware FP64 split (per-row weights for A, per-column for B): the form of
Eq. (ozakiscaled) with stored power-of-two weights that the paper names as its
key future step (Sec. 9).  Pins: properties the weights must give exactly
(power-of-two invariance, reduction to the paper's operand-wide split), the
widened input domain, and the accuracy it recovers on scaled rows."""
import numpy as np
import pytest

import oracle as O
import seeded_inputs as S


def test_scale_exponents_definition():
    X = np.array([[0.0, 0.0, 0.0], [1.0, -0.5, 0.25], [0.75, 0.1, -0.2],
                  [-3.0, 2.0, 1.0], [2.0 ** -300, 0.0, 0.0], [np.inf, 1.5, 0.0]])
    # ceil(log2 max|x|): 0 for an empty row; 1 -> 0; 0.75 -> 0; 3 -> 2; 2^-300 -> -300;
    # non-finite entries are ignored (1.5 -> 1)
    assert list(O.scale_exponents(X)) == [0, 0, 0, 2, -300, 1]
    assert list(O.scale_exponents(X.T, by_col=True)) == [0, 0, 0, 2, -300, 1]


@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
def test_power_of_two_row_and_column_weights_factor_out_exactly(nprod):
    """Multiplying row m of A by 2^e_m and column n of B by 2^f_n multiplies
    C_mn by exactly 2^(e_m + f_n) in the scale-aware form."""
    rng = np.random.default_rng(nprod)
    A = S.make("uniform", 501, (37, 300), np.float64)
    B = S.make("wide", 502, (300, 29), np.float64)
    e = rng.integers(-60, 61, 37)
    f = rng.integers(-60, 61, 29)
    C, st = O.emu_dgemm(A, B, nprod, scope=O.SCOPE_ROWCOL)
    C2, st2 = O.emu_dgemm(np.ldexp(A, e[:, None]), np.ldexp(B, f[None, :]), nprod,
                          scope=O.SCOPE_ROWCOL)
    assert st == 0 and st2 == 0
    assert np.array_equal(C2, np.ldexp(C, e[:, None] + f[None, :]))


@pytest.mark.parametrize("nprod", [6, 21])
def test_reduces_to_operand_wide_split_when_rows_share_a_binade(nprod):
    """If every row of A and every column of B has its maximum in the binade of
    the operand's maximum, the weights are one common power of two and the
    result is the paper's operand-wide result, bit for bit."""
    A = S.make("uniform", 511, (30, 260), np.float64)
    B = S.make("uniform", 512, (260, 20), np.float64)
    A[:, 0] = 0.9375                 # every row max in (1/2, 1]
    B[0, :] = -0.875                 # every column max in (1/2, 1]
    assert set(O.scale_exponents(A)) == {0} and set(O.scale_exponents(B, True)) == {0}
    C0, _ = O.emu_dgemm(A, B, nprod)
    C1, _ = O.emu_dgemm(A, B, nprod, scope=O.SCOPE_ROWCOL)
    assert np.array_equal(C0, C1)


def test_domain_extends_beyond_the_bf16_exponent_range():
    """Entries around 1e200 and 1e-200 lie outside the BF16 range of Eq.
    (bf16rangefp64): the operand-wide split flags them; with per-row and
    per-column weights the split is in range and the result keeps FP64-level
    accuracy."""
    A = S.make("uniform", 521, (24, 200), np.float64) * 1e200
    B = S.make("uniform", 522, (200, 18), np.float64) * 1e-200
    _, st_op = O.emu_dgemm(A, B, 21)
    assert st_op & O.ST_RANGE
    C, st = O.emu_dgemm(A, B, 21, scope=O.SCOPE_ROWCOL)
    assert st == 0
    hi, _ = O.ref_gemm_dd(A, B)
    assert O.e_F(C, hi) < 4e-16


def test_recovers_accuracy_lost_to_scaled_rows():
    """1 % of the rows of A scaled by 2^16 (B unscaled): with operand-wide
    exponents the other rows lose 16 bits in every slice; with row weights the
    error returns to that of the unscaled problem."""
    A0 = S.make("normal", 531, (200, 256), np.float64)
    B = S.make("normal", 532, (256, 64), np.float64)
    A = A0.copy()
    A[::100] *= 2.0 ** 16
    ref0, _ = O.ref_gemm_dd(A0, B)
    ref, _ = O.ref_gemm_dd(A, B)
    base, _ = O.emu_dgemm(A0, B, 10)
    opw, _ = O.emu_dgemm(A, B, 10)
    rc, st = O.emu_dgemm(A, B, 10, scope=O.SCOPE_ROWCOL)
    assert st == 0
    keep = np.ones(A.shape[0], bool)
    keep[::100] = False
    e_base = O.e_F(base[keep], ref0[keep])
    e_op, e_rc = O.e_F(opw[keep], ref[keep]), O.e_F(rc[keep], ref[keep])
    assert e_op > 100 * e_base, (e_op, e_base)
    assert e_rc < 2 * e_base, (e_rc, e_base)


def test_entries_follow_the_full_scaled_gemm():
    A = S.make("normal_scaled_rows", 541, (150, 300), np.float64)
    B = S.make("wide", 542, (300, 70), np.float64)
    C, _ = O.emu_dgemm(A, B, 15, scope=O.SCOPE_ROWCOL)
    r = np.array([0, 149, 3, 77, 100])
    c = np.array([0, 69, 50, 1, 33])
    e, _ = O.emu_dgemm_entries(A, B, r, c, 15, scope=O.SCOPE_ROWCOL)
    assert np.array_equal(e, C[r, c])
