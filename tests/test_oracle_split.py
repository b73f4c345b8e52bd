"""Pins of the oracle's component splits against the paper and the mathematics.

FP32 split: Eq. (fp32split), Sec. 4.2 (three BF16 components, residuals exact by
Sterbenz's lemma).  FP64 split: Eq. (fp64split), Sec. 4.3 (fixed six slices,
operand-wide v = ceil(log2 max|A^(r)|), add-subtract projection with rho = 45,
zero-residual rule).  Nothing here calls the oracle's arithmetic to produce an
expected value: expectations come from exact rational arithmetic, an
independent integer form of round-to-nearest-even, or closed forms.
"""
import math
import os
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import seeded_inputs as S
from _exact import bf16_value, ceil_log2, f32_bits, to_bf16

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


# ---------------------------------------------------------------------------
# BF16 rounding


def test_bf16_rne_f32_definition_samples():
    # ties: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> even (1.0)
    assert O.bf16_rne_f32(1.0 + 2.0 ** -8) == 0x3F80
    # 1 + 3*2^-8 is halfway between 1+2^-7 (odd) and 1+2^-6 (even) -> 1+2^-6
    assert O.bf16_rne_f32(1.0 + 3 * 2.0 ** -8) == 0x3F82
    assert O.bf16_rne_f32(-(1.0 + 3 * 2.0 ** -8)) == 0xBF82
    # just above a tie rounds up
    assert O.bf16_rne_f32(np.float32(1.0 + 2.0 ** -8 + 2.0 ** -20)) == 0x3F81
    # overflow of the largest binary32 -> +inf
    assert O.bf16_rne_f32(np.float32(3.4028234663852886e38)) == 0x7F80
    # largest value that still rounds to the largest finite BF16
    assert O.bf16_rne_f32(np.float32((2 - 2.0 ** -7 + 2.0 ** -9) * 2.0 ** 127)) == 0x7F7F


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_bf16_rne_f64_against_fractions(seed):
    rng = np.random.default_rng(seed)
    vals = np.concatenate([
        rng.standard_normal(300) * 2.0 ** rng.integers(-140, 130, 300),
        [0.0, -0.0, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 2.0 ** -126 * (1 - 2.0 ** -9)],
        # a detour through binary32 would round these twice: first onto the
        # BF16 midpoint, then to even; one rounding goes the other way
        [1 + 2.0 ** -8 + 2.0 ** -30, -(1 + 2.0 ** -8 + 2.0 ** -30), 1 + 3 * 2.0 ** -8 - 2.0 ** -30,
         (1 + 2.0 ** -8 + 2.0 ** -40) * 2.0 ** 50],
    ])
    for x in vals:
        h = O.bf16_rne_f64(float(x))
        ref = to_bf16(Fraction(float(x)))
        if isinstance(ref, float):
            assert (h & 0x7FFF) == 0x7F80
        else:
            assert bf16_value(h) == ref, (x, hex(h))


# ---------------------------------------------------------------------------
# FP32 split


@pytest.mark.slow
def test_split_f32_exhaustive_all_bit_patterns(tmp_path):
    """Every finite binary32 a with 2^-103 <= |a| < (2-2^-8) 2^127, and +-0,
    splits exactly into three normal-or-zero BF16 components; A_0 is RNE."""
    O.build(force=False)
    exe = str(tmp_path / "exh")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off",
                    os.path.join(ROOT, "tests", "csrc", "exhaustive_split32.c"),
                    "-L" + os.path.join(ROOT, "oracle"), "-loracle",
                    "-Wl,-rpath," + os.path.join(ROOT, "oracle"), "-lm", "-o", exe], check=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split()
    n_finite, n_in, bad_in, rne_bad, fail_out, fail_low, fail_high = map(int, out)
    assert n_finite == 2 ** 32 - 2 * 2 ** 23          # all but NaN/Inf patterns
    assert bad_in == 0
    assert rne_bad == 0
    assert n_in > 0 and fail_out == fail_low + fail_high
    # failures exist only below the range (subnormal tails) and in the a0-overflow band
    assert fail_low > 0 and fail_high == 2 * 2 ** 15


def test_split_f32_residual_shrinks_by_u_bf16():
    """Each residual step shrinks the magnitude by at most u_BF16 = 2^-8 relative
    to the value it was extracted from (Sec. 4.2)."""
    X = S.make("normal", 11, (64, 97), np.float32)
    c, st = O.split_f32(X)
    assert st == 0
    a0, a1, a2 = (O.bf16_to_f32(c[t]).astype(np.float64) for t in range(3))
    x = X.astype(np.float64)
    r1 = x - a0
    r2 = r1 - a1
    assert np.all(np.abs(r1) <= np.abs(x) * 2.0 ** -8)
    assert np.all(np.abs(r2) <= np.abs(r1) * 2.0 ** -8)
    assert np.array_equal(a0 + a1 + a2, x)


def test_split_f32_flags():
    X = np.array([[np.nan, 1.0], [3.4028234663852886e38, 1e-44]], dtype=np.float32)
    _, st = O.split_f32(X)
    assert st & O.ST_NAN
    assert st & O.ST_OVERFLOW
    assert st & O.ST_SUBNORMAL


# ---------------------------------------------------------------------------
# FP64 split


def _check_split_f64_exact(X, mode):
    """Check every stated property of Eq. (fp64split) with exact rationals."""
    slices, v, resid, st = O.split_f64(X, mode)
    R, C = X.shape
    W = [[Fraction(float(X[i, j])) for j in range(C)] for i in range(R)]
    done = False
    for r in range(6):
        m = max(abs(w) for row in W for w in row)
        if m == 0 or done:
            done = True
            assert v[r] == np.iinfo(np.int32).min
            assert not slices[r].any()
            continue
        vr = ceil_log2(m)
        assert v[r] == vr, (r, v[r], vr)
        if r > 0 and mode == O.SPLIT_SYM:
            assert v[r] <= v[r - 1] - 9
        unit_neg = Fraction(2) ** (vr - 8)
        unit_pos = Fraction(2) ** (vr - 7) if mode == O.SPLIT_LITERAL else unit_neg
        for i in range(R):
            for j in range(C):
                w = W[i][j]
                z = bf16_value(slices[r, i, j])
                unit = unit_pos if w >= 0 else unit_neg
                # Z is the nearest multiple of the unit, ties to even
                q = w / unit
                n = math.floor(q)
                rem = q - n
                if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2):
                    n += 1
                assert z == n * unit, (r, i, j)
                assert abs(z) <= Fraction(2) ** vr
                W[i][j] = w - z                       # exact residual update
    for i in range(R):
        for j in range(C):
            total = sum(bf16_value(slices[r, i, j]) for r in range(6))
            assert total + Fraction(float(resid[i, j])) == Fraction(float(X[i, j]))
            assert Fraction(float(resid[i, j])) == W[i][j]
    if mode == O.SPLIT_SYM and v[5] != np.iinfo(np.int32).min:
        assert np.all(np.abs(resid) <= 2.0 ** (int(v[5]) - 9))
    return slices, v, st


@pytest.mark.parametrize("mode", [O.SPLIT_SYM, O.SPLIT_LITERAL])
@pytest.mark.parametrize("dist", ["uniform", "normal", "wide"])
def test_split_f64_exact_properties(mode, dist):
    X = S.make(dist, 21, (5, 7), np.float64)
    _, _, st = _check_split_f64_exact(X, mode)
    assert st == 0


def test_split_f64_adversarial():
    X = np.array([[1.0, -1.0, 0.5], [2.0 ** -20, 3.0, -0.75]])        # max a power of two? (3)
    _check_split_f64_exact(X, O.SPLIT_SYM)
    X = np.array([[4.0, -1.0], [0.5, 4.0 - 2.0 ** -40]])               # max just below 2^2
    _check_split_f64_exact(X, O.SPLIT_SYM)
    X = np.array([[2.0 ** -70, -3 * 2.0 ** -72], [2.0 ** -71, 0.0]])   # tiny operand max
    _, _, st = _check_split_f64_exact(X, O.SPLIT_SYM)
    assert st == 0


def test_split_f64_zero_and_single_nonzero():
    Z = np.zeros((3, 4))
    slices, v, resid, st = O.split_f64(Z)
    assert st == 0 and not slices.any() and not resid.any()
    assert all(x == np.iinfo(np.int32).min for x in v)
    X = np.zeros((3, 4))
    X[1, 2] = 1.0 / 3.0
    slices, v, _ = _check_split_f64_exact(X, O.SPLIT_SYM)
    assert list(v) == [-1, -10, -19, -28, -37, -46]


def test_split_f64_bf16_exact_matrix_has_one_slice():
    rng = np.random.default_rng(5)
    h = rng.integers(0, 0x7F, (8, 9)).astype(np.uint16) | np.uint16(0x3F00)
    X = O.bf16_to_f32(h).astype(np.float64) * rng.choice([-1.0, 1.0], (8, 9))
    slices, v, resid, st = O.split_f64(X)
    # Every entry is a multiple of 2^(v0-8) when all entries share the top binade.
    assert st == 0 and not slices[1:].any() and not resid.any()
    assert np.array_equal(O.bf16_to_f32(slices[0]).astype(np.float64), X)


def test_split_f64_integer_matrix_two_slices():
    rng = np.random.default_rng(6)
    X = rng.integers(-2 ** 15, 2 ** 15 + 1, (16, 16)).astype(np.float64)
    X[0, 0] = 2.0 ** 15
    slices, v, resid, st = O.split_f64(X)
    assert st == 0 and v[0] == 15 and not slices[2:].any() and not resid.any()


def test_split_f64_domain_flags():
    _, _, _, st = O.split_f64(np.array([[1.0, np.inf]]))
    assert st & O.ST_NAN
    _, _, _, st = O.split_f64(np.array([[1.0, 2.0 ** -130]]))
    assert st & O.ST_RANGE
    _, _, _, st = O.split_f64(np.array([[2.0 ** 200, 1.0]]))
    assert st & O.ST_RANGE
    # operand max near the bottom of the BF16 range: lower slices become subnormal
    _, _, _, st = O.split_f64(np.array([[2.0 ** -120 * (1 + 2.0 ** -30), 2.0 ** -121]]))
    assert st & O.ST_SUBNORMAL


def test_split_f64_uniform_chain_is_nine_bits_per_level():
    """For uniform[-1,1] operands the sym split keeps 9 bits per level:
    v_r = -9 r (the residual max fills each half-unit)."""
    X = S.make("uniform", 3001, (256, 256), np.float64)
    _, v, _, st = O.split_f64(X)
    assert st == 0
    assert list(v) == [0, -9, -18, -27, -36, -45]
