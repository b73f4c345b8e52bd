"""Pins of the oracle's emulated GEMMs and references.

Emulated SGEMM: Algorithm fp32, Eq. (fp32six), executed per reduction panel of
length B_K = 256 in the operand-reuse order of Eq. (fp32reuseorder) (Sec. 6.2,
6.3).  Emulated DGEMM: Algorithm fp64, Eq. (fp64reconstruction), per panel,
diagonals ascending, i ascending inside a diagonal (Sec. 6.3).

Pins (none of them re-run the oracle's own arithmetic):
  * integer inputs whose products the retained set captures exactly -> C = AB;
  * B = I closed forms;
  * tiny shapes against an exact-rational (Fraction) evaluation of the
    definition;
  * the accuracy values the paper prints (Sec. 8.2, tests/golden);
  * the closed form e_F(d) ~ sqrt(n_d) 2^(-9d) for uniform inputs;
  * error bounds of the double-double reference.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import seeded_inputs as S
from _exact import bf16_value, to_f32

HERE = os.path.dirname(os.path.abspath(__file__))
REUSE = [(1, 1), (1, 0), (2, 0), (0, 0), (0, 1), (0, 2)]


def _round64(x: Fraction) -> Fraction:
    return Fraction(float(x))          # Python's float(Fraction) rounds correctly, ties even


def _f32(x: Fraction) -> Fraction:
    r = to_f32(x)
    assert not isinstance(r, float)
    return r


# ---------------------------------------------------------------------------
# integer and identity pins


def test_sgemm_bf16_exact_integers_give_exact_product():
    rng = np.random.default_rng(1)
    A = rng.integers(-256, 257, (7, 256)).astype(np.float32)
    B = rng.integers(-256, 257, (256, 9)).astype(np.float32)
    C, st = O.emu_sgemm(A, B)
    exact = A.astype(np.int64) @ B.astype(np.int64)
    assert st == 0 and np.array_equal(C.astype(np.int64), exact)


def test_sgemm_cross_products_integers():
    """|x| <= 1000 needs two BF16 components; A0B0, A0B1, A1B0 and A1B1 are all
    nonzero and every partial sum is an integer below 2^24, so C = AB."""
    rng = np.random.default_rng(2)
    A = rng.integers(-1000, 1001, (11, 16)).astype(np.float32)
    B = rng.integers(-1000, 1001, (16, 13)).astype(np.float32)
    c, _ = O.split_f32(A)
    assert c[1].any() and not c[2].any()
    C, st = O.emu_sgemm(A, B)
    exact = A.astype(np.int64) @ B.astype(np.int64)
    assert np.array_equal(C.astype(np.int64), exact)


def test_sgemm_identity_reconstructs_input():
    A = S.make("normal", 7, (37, 300), np.float32)
    C, st = O.emu_sgemm(A, np.eye(300, dtype=np.float32))
    assert st == 0 and np.array_equal(C, A)


@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
def test_dgemm_integers_give_exact_product(nprod):
    rng = np.random.default_rng(3)
    A = rng.integers(-2 ** 15, 2 ** 15 + 1, (9, 600)).astype(np.float64)
    B = rng.integers(-2 ** 15, 2 ** 15 + 1, (600, 7)).astype(np.float64)
    C, st = O.emu_dgemm(A, B, nprod)
    exact = A.astype(np.int64) @ B.astype(np.int64)
    assert st == 0 and np.array_equal(C.astype(np.int64), exact)


@pytest.mark.parametrize("nprod", [1, 3, 6, 10, 15, 21, 26, 36])
def test_dgemm_identity_sums_retained_slices(nprod):
    d = O.NPROD_TO_D[nprod]
    A = S.make("uniform", 8, (5, 260), np.float64)
    C, st = O.emu_dgemm(A, np.eye(260), nprod)
    slices, _, resid, _ = O.split_f64(A)
    for i in range(5):
        for j in range(260):
            c = Fraction(0)
            for r in range(min(d, 6)):              # products (r, 0), diagonal r
                c = _round64(c + bf16_value(slices[r, i, j]))
            assert Fraction(float(C[i, j])) == c
    if d >= 6:
        assert np.array_equal(C, A - resid) or np.max(np.abs(C - (A - resid))) <= 2.0 ** -53


def test_degenerate_sizes():
    C, _ = O.emu_sgemm(np.zeros((3, 0), np.float32), np.zeros((0, 4), np.float32))
    assert C.shape == (3, 4) and not C.any()
    C, _ = O.emu_dgemm(np.zeros((3, 0)), np.zeros((0, 4)), 10)
    assert C.shape == (3, 4) and not C.any()


# ---------------------------------------------------------------------------
# brute force against exact rationals


@pytest.mark.parametrize("shape", [(3, 5, 4), (2, 3, 300)])
def test_sgemm_definition_bruteforce(shape):
    M, N, K = shape
    A = S.make("normal", 31, (M, K), np.float32)
    B = S.make("wide", 32, (K, N), np.float32)
    C, _ = O.emu_sgemm(A, B)
    ca, _ = O.split_f32(A)
    cb, _ = O.split_f32(B)
    for m in range(M):
        for n in range(N):
            blk = Fraction(0)
            for p0 in range(0, K, 256):
                t = Fraction(0)
                for i, j in REUSE:
                    P = sum(bf16_value(ca[i, m, k]) * bf16_value(cb[j, k, n])
                            for k in range(p0, min(K, p0 + 256)))
                    t = _f32(t + _f32(P))
                blk = _f32(blk + t)
            assert Fraction(float(C[m, n])) == blk, (m, n)


@pytest.mark.parametrize("nprod", [1, 3, 6, 21, 30, 36])
@pytest.mark.parametrize("shape", [(3, 4, 5), (2, 3, 520)])
def test_dgemm_definition_bruteforce(nprod, shape):
    M, N, K = shape
    d = O.NPROD_TO_D[nprod]
    A = S.make("wide", 41, (M, K), np.float64)
    B = S.make("uniform", 42, (K, N), np.float64)
    C, st = O.emu_dgemm(A, B, nprod)
    assert st == 0
    sa, _, _, _ = O.split_f64(A)
    sb, _, _, _ = O.split_f64(B)
    for m in range(M):
        for n in range(N):
            c = Fraction(0)
            for p0 in range(0, K, 256):
                for ell in range(d):
                    for i in range(max(0, ell - 5), min(ell, 5) + 1):
                        j = ell - i
                        P = sum(bf16_value(sa[i, m, k]) * bf16_value(sb[j, k, n])
                                for k in range(p0, min(K, p0 + 256)))
                        assert _f32(P) == P            # panel products are exact in FP32
                        c = _round64(c + P)
            assert Fraction(float(C[m, n])) == c, (m, n)


@pytest.mark.parametrize("nprod", [21, 36])
def test_dgemm_definition_bruteforce_order_sensitive(nprod):
    """K = 1 and 21 or all 36 products: the FP64 chain spans more than 53 bits,
    so the roundings of the last diagonals depend on the order of the additions
    (diagonal ascending, i ascending): 4096 entries against exact products
    added in that order in Python floats (IEEE binary64)."""
    d = O.NPROD_TO_D[nprod]
    A = S.make("wide", 43, (64, 1), np.float64)
    B = S.make("wide", 44, (1, 64), np.float64)
    C, st = O.emu_dgemm(A, B, nprod)
    assert st == 0
    sa, _, _, _ = O.split_f64(A)
    sb, _, _, _ = O.split_f64(B)
    av = np.vectorize(lambda h: float(bf16_value(h)))(sa[:, :, 0])    # [6, 64]
    bv = np.vectorize(lambda h: float(bf16_value(h)))(sb[:, 0, :])    # [6, 64]
    for m in range(64):
        for n in range(64):
            c = 0.0
            for ell in range(d):
                for i in range(max(0, ell - 5), min(ell, 5) + 1):
                    c = c + av[i, m] * bv[ell - i, n]     # exact product (<= 16 bits)
            assert C[m, n] == c, (m, n)


def test_dot_bf16_f32_ties_to_even():
    """Exact sums halfway between two binary32 values round to the even one."""
    one, tiny = 0x3F80, 0x3380                     # BF16 1.0 and 2^-24
    three_tiny = 0x3440                            # 3 * 2^-24
    cases = [([one, tiny], 1.0),                   # 1 + 2^-24 -> 1
             ([one, three_tiny], 1.0 + 2.0 ** -22),   # 1 + 3 2^-24 -> 1 + 2^-22
             ([0xBF80, 0xB380], -1.0)]             # sign symmetric
    for xs, want in cases:
        x = np.array(xs, dtype=np.uint16)
        y = np.array([one, one], dtype=np.uint16)
        assert bf16_value(x[1]) in (Fraction(1, 2 ** 24), Fraction(3, 2 ** 24), Fraction(-1, 2 ** 24))
        assert O.dot_bf16_f32(x, y) == want, (xs, want)


def test_dot_bf16_f32_correct_rounding_wide_range():
    rng = np.random.default_rng(9)
    for trial in range(40):
        n = int(rng.integers(1, 300))
        ex = rng.integers(1, 254, (2, n))
        if trial % 4 == 0:
            ex[:, ::7] = 0                           # include BF16 subnormals
        fr = rng.integers(0, 128, (2, n))
        sg = rng.integers(0, 2, (2, n))
        h = ((sg << 15) | (ex << 7) | fr).astype(np.uint16)
        got = O.dot_bf16_f32(h[0], h[1])
        exact = sum(bf16_value(h[0, k]) * bf16_value(h[1, k]) for k in range(n))
        ref = to_f32(exact)
        if isinstance(ref, float):
            assert math.isinf(got) and (got > 0) == (ref > 0)
        else:
            assert Fraction(got) == ref


# ---------------------------------------------------------------------------
# values printed in the paper, and closed forms


def _golden():
    with open(os.path.join(HERE, "golden", "table_accuracy.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("n", [256, 512])
def test_table_accuracy_fp64_columns(n):
    """Sec. 8.2, Table accuracy, uniform[-1,1]: e_F and e_scaled of the FP64
    variants against a DGEMM result.  A plain FP64 GEMM stands in for oneMKL
    DGEMM (its own error only matters for the 21-product column)."""
    row = _golden()["rows"][str(n)]
    A = S.make("uniform", 3001, (n, n), np.float64)
    B = S.make("uniform", 3002, (n, n), np.float64)
    ref = O.ref_gemm_f64(A, B)
    ab = np.abs(A) @ np.abs(B)
    for col, nprod in enumerate((6, 10, 15, 21), start=1):
        C, st = O.emu_dgemm(A, B, nprod)
        assert st == 0
        eF = O.e_F(C, ref)
        esc, _ = O.e_scaled(C, ref, ab)
        if nprod < 21:
            assert abs(eF / row["e_F"][col] - 1) < 0.05, (nprod, eF)
            assert 1 / 1.5 < esc / row["e_scaled"][col] < 1.5, (nprod, esc)
        else:
            assert 0.5 < eF / row["e_F"][col] < 2.0, (nprod, eF)
            assert 0.5 < esc / row["e_scaled"][col] < 2.0, (nprod, esc)


@pytest.mark.parametrize("n", [256, 512])
def test_table_accuracy_fp32_column(n):
    """FP32 column against an SGEMM result: numpy's FP32 matmul stands in for
    oneMKL SGEMM; its own error is part of the printed number."""
    row = _golden()["rows"][str(n)]
    A = S.make("uniform", 1001, (n, n), np.float32)
    B = S.make("uniform", 1002, (n, n), np.float32)
    C, st = O.emu_sgemm(A, B)
    sg = (A @ B).astype(np.float64)
    ab = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    eF = O.e_F(C, sg)
    esc, _ = O.e_scaled(C, sg, ab)
    assert abs(eF / row["e_F"][0] - 1) < 0.15, eF
    assert 1 / 1.5 < esc / row["e_scaled"][0] < 1.5, esc
    # against an exact reference the emulation itself is well below FP32 level
    assert O.e_F(C, O.ref_gemm_f64(A, B)) < 1.0e-7


def test_closed_form_uniform_fp64_error():
    """With nine bits per level, slice i of a uniform operand has standard
    deviation 2^(-9i) times that of the operand, so the first omitted diagonal
    gives e_F(d) ~ sqrt(n_d) 2^(-9d), n_d = number of pairs on diagonal d."""
    n = 384
    A = S.make("uniform", 3001, (n, n), np.float64)
    B = S.make("uniform", 3002, (n, n), np.float64)
    ref = O.ref_gemm_dd(A, B)
    for nprod, d in ((6, 3), (10, 4), (15, 5)):
        C, _ = O.emu_dgemm(A, B, nprod)
        pred = math.sqrt(d + 1) * 2.0 ** (-9 * d)
        assert abs(O.e_F(C, ref) / pred - 1) < 0.05, nprod
    C, _ = O.emu_dgemm(A, B, 21)
    assert O.e_F(C, ref) < 4e-16


def test_literal_projection_does_not_match_table():
    """The literal constant 2^(v+45) keeps about one bit less per level for
    non-negative residuals; its FP64-6 error is far above the printed 1.49e-8."""
    A = S.make("uniform", 3001, (256, 256), np.float64)
    B = S.make("uniform", 3002, (256, 256), np.float64)
    C, _ = O.emu_dgemm(A, B, 6, mode=O.SPLIT_LITERAL)
    assert O.e_F(C, O.ref_gemm_dd(A, B)) > 3 * 1.49e-8


# ---------------------------------------------------------------------------
# references and entry sampling


def test_dd_reference_error_bound():
    rng = np.random.default_rng(4)
    A = rng.standard_normal((4, 50)) * 2.0 ** rng.integers(-30, 30, (4, 50))
    B = rng.standard_normal((50, 3))
    hi, lo = O.ref_gemm_dd(A, B)
    u = 2.0 ** -53
    for m in range(4):
        for n in range(3):
            exact = sum(Fraction(float(A[m, k])) * Fraction(float(B[k, n])) for k in range(50))
            absum = sum(abs(Fraction(float(A[m, k])) * Fraction(float(B[k, n]))) for k in range(50))
            err = abs(Fraction(float(hi[m, n])) + Fraction(float(lo[m, n])) - exact)
            assert err <= 2 * 50 ** 2 * Fraction(u) ** 2 * absum + Fraction(u) ** 2 * abs(exact)


def test_entries_match_full_gemm():
    A = S.make("normal", 51, (40, 300), np.float64)
    B = S.make("normal", 52, (300, 33), np.float64)
    rows = np.array([0, 5, 39, 17])
    cols = np.array([0, 32, 7, 7])
    C, _ = O.emu_dgemm(A, B, 15)
    e, _ = O.emu_dgemm_entries(A, B, rows, cols, 15)
    assert np.array_equal(e, C[rows, cols])
    A32, B32 = A.astype(np.float32), B.astype(np.float32)
    C32, _ = O.emu_sgemm(A32, B32)
    e32, _ = O.emu_sgemm_entries(A32, B32, rows, cols)
    assert np.array_equal(e32, C32[rows, cols])
    hi, lo = O.ref_gemm_dd(A, B)
    h2, l2 = O.ref_dd_entries(A, B, rows, cols)
    assert np.array_equal(h2, hi[rows, cols]) and np.array_equal(l2, lo[rows, cols])
    ab = O.absprod_entries(A, B, rows, cols)
    assert np.allclose(ab, (np.abs(A) @ np.abs(B))[rows, cols], rtol=1e-14)


# ---------------------------------------------------------------------------
# the inexact-panel status bit (16): a panel product that is not an FP32 value


def _inexact_by_definition(A, B, nprod, kc):
    """Whether some exact panel sum of a retained product is not a binary32
    value (Fractions over the oracle's own slices, which the split pins fix)."""
    d = O.NPROD_TO_D[nprod]
    sa, _, _, _ = O.split_f64(A)
    sb, _, _, _ = O.split_f64(B)
    M, K = A.shape
    N = B.shape[1]
    av = [[[bf16_value(sa[i, m, k]) for k in range(K)] for m in range(M)] for i in range(6)]
    bv = [[[bf16_value(sb[j, k, n]) for k in range(K)] for n in range(N)] for j in range(6)]
    for m in range(M):
        for n in range(N):
            for p0 in range(0, K, kc):
                for ell in range(d):
                    for i in range(max(0, ell - 5), min(ell, 5) + 1):
                        j = ell - i
                        P = sum(av[i][m][k] * bv[j][n][k] for k in range(p0, min(K, p0 + kc)))
                        r = to_f32(P)
                        if isinstance(r, float) or r != P:
                            return True
    return False


def test_dgemm_inexact_panel_flag_long_panel():
    """Slice entries of 255 units: 256 of them stay below 2^24 units (exact),
    511 in one panel reach 511 * 255^2 > 2^24, an odd number of units that
    binary32 cannot hold.  Panels of 512 must raise bit 16 and lose the exact
    product; panels of 256 give it exactly with no flag."""
    K = 511
    A = np.full((2, K), 255.0 / 256.0)
    B = np.full((K, 2), 255.0 / 256.0)
    exact = Fraction(K) * Fraction(255, 256) ** 2
    assert _inexact_by_definition(A, B, 6, 512) and not _inexact_by_definition(A, B, 6, 256)
    C, st = O.emu_dgemm(A, B, 6, kc=512)
    assert st & O.ST_INEXACT32 and Fraction(float(C[0, 0])) != exact
    C, st = O.emu_dgemm(A, B, 6)
    assert st == 0 and np.all(C == float(exact))


@pytest.mark.parametrize("scale", [0, -30, -45])
@pytest.mark.parametrize("nprod", [6, 15, 21])
def test_dgemm_inexact_flag_matches_definition(scale, nprod):
    """Tiny operands push the lower panel products below FP32's subnormal
    spacing: the flag is raised exactly when some panel sum, computed with
    exact rationals, is not a binary32 value."""
    A = np.ldexp(S.make("uniform", 51, (2, 40), np.float64), scale)
    B = np.ldexp(S.make("uniform", 52, (40, 2), np.float64), scale)
    _, st = O.emu_dgemm(A, B, nprod)
    assert bool(st & O.ST_INEXACT32) == _inexact_by_definition(A, B, nprod, 256)
    assert (st & ~O.ST_INEXACT32) == 0


def test_dgemm_inexact_flag_cases_are_not_vacuous():
    A = np.ldexp(S.make("uniform", 51, (2, 40), np.float64), -45)
    B = np.ldexp(S.make("uniform", 52, (40, 2), np.float64), -45)
    assert _inexact_by_definition(A, B, 21, 256) and not _inexact_by_definition(A, B, 6, 256)


def test_entries_from_presplit_components_match():
    """The benchmark's pre-split entry points give the bits of the plain ones."""
    A = S.make("wide", 61, (9, 300), np.float64)
    B = S.make("uniform", 62, (300, 7), np.float64)
    rows = np.array([0, 3, 8, 8], np.int64)
    cols = np.array([0, 6, 1, 6], np.int64)
    sa, _, _, _ = O.split_f64(A)
    sb, _, _, _ = O.split_f64(B)
    for nprod in (6, 21, 36):
        want, st = O.emu_dgemm_entries(A, B, rows, cols, nprod)
        got, st2 = O.dgemm_entries_from_slices(sa, sb, rows, cols, nprod)
        assert st == st2 == 0 and np.array_equal(got.view(np.uint64), want.view(np.uint64))
    A32, B32 = A.astype(np.float32), B.astype(np.float32)
    want, _ = O.emu_sgemm_entries(A32, B32, rows, cols)
    got = O.sgemm_entries_from_comps(O.split_f32(A32)[0], O.split_f32(B32)[0], rows, cols)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
