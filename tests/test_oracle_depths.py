"""Pins of the oracle's emulated DGEMM at every depth of the triangular product
selection, Eq. (product-selection): S_d = {(i, j) : 0 <= i, j < 6, i + j < d}
for d = 1 .. 11 (d = 11 keeps all 36 products; the paper evaluates d = 3 .. 6,
Eq. fp64productcounts, and names the full 6 x 6 set as the limit, Sec. 4.3).

None of these re-run the oracle's arithmetic: the product counts are closed
forms, the structured operands below have slices fixed by hand from the
projection of Eq. (fp64split), and the error of uniform inputs follows the
nine-bits-per-level closed form.
"""
import math

import numpy as np
import pytest

import oracle as O
import seeded_inputs as S

DEPTHS = range(1, 12)


def n_p(d):
    """|S_d| in closed form: d (d + 1) / 2 up to d = 6, then 36 minus the
    untouched triangle (11 - d)(12 - d) / 2."""
    return d * (d + 1) // 2 if d <= 6 else 36 - (11 - d) * (12 - d) // 2


def test_product_counts():
    assert [n_p(d) for d in DEPTHS] == [1, 3, 6, 10, 15, 21, 26, 30, 33, 35, 36]
    assert O.NPROD_TO_D == {n_p(d): d for d in DEPTHS}


@pytest.mark.parametrize("nprod", [0, 2, 4, 7, 20, 22, 34, 37, -6])
def test_other_product_counts_rejected(nprod):
    A = np.ones((2, 3))
    C = np.zeros((2, 2))
    L = O.lib()
    st = L.orc_emu_dgemm(2, 2, 3, A.ctypes.data, 3, np.ones((3, 2)).ctypes.data, 2,
                         C.ctypes.data, 2, nprod, O.SPLIT_SYM, O.KC)
    assert st == 0xFFFFFFFF


# Structured operands (K = 1).  A = [a; x], B = [b, y] with
#   a = b = 1 + 2^-9 + 2^-18 + 2^-27 + 2^-36,   x = y = 2^-60.
# Level by level (v_r = ceil(log2 max|residual|), unit 2^(v_r - 8)):
#   r = 0: v = 1, a_0 = 1, x_0 = 0;  r = 1..4: v = -8, -17, -26, -36 and
#   a_r = 2^(-9 r), x_r = 0 (2^-60 is below half a unit);  r = 5: a's residual
#   is 0, so v_5 = -60 and x_5 = 2^-60.
# Hence a_i b_j = 2^(-9 (i + j)) for i, j <= 4, x b_j = 2^(-60 - 9 j) through
# (5, j) only, and x y through (5, 5) only.
A_VAL = sum(2.0 ** (-9 * i) for i in range(5))
X_VAL = 2.0 ** -60


def test_structured_operands_split_as_stated():
    slices, v, _, st = O.split_f64(np.array([[A_VAL], [X_VAL]]))
    assert st == 0 and list(v) == [1, -8, -17, -26, -36, -60]
    from _exact import bf16_value
    got = [[float(bf16_value(slices[r, m, 0])) for r in range(6)] for m in range(2)]
    assert got[0] == [2.0 ** (-9 * r) for r in range(5)] + [0.0]
    assert got[1] == [0.0] * 5 + [X_VAL]


@pytest.mark.parametrize("d", DEPTHS)
def test_structured_operands_closed_form(d):
    A = np.array([[A_VAL], [X_VAL]])
    B = np.array([[A_VAL, X_VAL]])
    C, st = O.emu_dgemm(A, B, n_p(d))
    assert st == 0
    # a b: diagonals l < min(d, 6) hold #{i + j = l, i, j <= 4} terms 2^(-9 l);
    # the partial sums span under 53 bits, and every later term (2^-54 and
    # below) is under half an ulp of the running sum, so it leaves it unchanged
    c00 = sum(sum(1 for i in range(5) if 0 <= l - i <= 4) * 2.0 ** (-9 * l)
              for l in range(min(d, 6)))
    # x b: products (5, j), j <= 4, retained when 5 + j < d (exact sum)
    c10 = sum(X_VAL * 2.0 ** (-9 * j) for j in range(5) if 5 + j < d)
    c11 = X_VAL * X_VAL if d == 11 else 0.0
    assert C[0, 0] == c00
    assert C[1, 0] == c10 and C[0, 1] == c10
    assert C[1, 1] == c11


def test_closed_form_uniform_low_depths():
    """d = 1, 2: the first omitted diagonal (d + 1 pairs of slices with
    standard deviation 2^(-9 d) relative) gives e_F ~ sqrt(d + 1) 2^(-9 d)."""
    n = 384
    A = S.make("uniform", 3001, (n, n), np.float64)
    B = S.make("uniform", 3002, (n, n), np.float64)
    ref = O.ref_gemm_f64(A, B)
    for d in (1, 2):
        C, _ = O.emu_dgemm(A, B, n_p(d))
        pred = math.sqrt(d + 1) * 2.0 ** (-9 * d)
        assert abs(O.e_F(C, ref) / pred - 1) < 0.05, d


def test_deep_depths_reach_fp64_level():
    """d >= 6 on uniform inputs: the omitted diagonals are below FP64 rounding,
    so e_F against the double-double reference stays at the d = 6 level."""
    n = 256
    A = S.make("uniform", 3101, (n, n), np.float64)
    B = S.make("uniform", 3102, (n, n), np.float64)
    ref = O.ref_gemm_dd(A, B)
    for d in range(6, 12):
        C, st = O.emu_dgemm(A, B, n_p(d))
        assert st == 0 and O.e_F(C, ref) < 4e-16, d
