"""Pins of the oracle's BLAS-form composition C = alpha op(A) op(B) + beta C.

The BLAS forms are the "more complete BLAS semantics" the paper names as
future work (Sec. 9).  The oracle composes them from its plain emulated GEMMs
(``_op``, ``_blas_out``, ``_scale_only``, ``emu_sgemm_ex``, ``emu_dgemm_ex`` in
``oracle/__init__.py``).  Each pin checks the composition against the BLAS
definition, not against the oracle's own code:

  * a transposed operand is the stored matrix read transposed: the result is
    the plain product of explicitly transposed copies, bit for bit;
  * alpha = 2^k with beta = 0 scales the product exactly (a power of two);
  * the update is fl(fl(alpha P) + fl(beta C)) in the output precision, two
    roundings and no fused multiply-add: checked with exact rationals on inputs
    chosen so that a fused or single-rounding update gives another value;
  * alpha = 0 or K = 0 gives beta C without reading A and B; beta = 0 never
    reads C.

The pins take the oracle module as an argument so that the mutation test at
the end can run them on copies of the module with a planted mistake.
"""
import os
import types
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import seeded_inputs as S
from _exact import round_nearest_even, to_f32

CASES = [("N", "N"), ("T", "N"), ("N", "T"), ("T", "T")]


def stored(X, trans):
    return np.ascontiguousarray(X.T) if trans == "T" else X


def to_f64(x: Fraction):
    return round_nearest_even(x, 53, -1022, 1023)


def pin_transposes(M):
    for (m, n, k) in ((7, 5, 300), (6, 6, 6)):
        A = S.make("wide", 801, (m, k), np.float64)
        B = S.make("uniform", 802, (k, n), np.float64)
        P, _ = M.emu_dgemm(A, B, 6)
        A32, B32 = A.astype(np.float32), B.astype(np.float32)
        P32, _ = M.emu_sgemm(A32, B32)
        for ta, tb in CASES:
            got, _ = M.emu_dgemm_ex(stored(A, ta), stored(B, tb), 6, None, ta, tb)
            assert got.shape == P.shape and np.array_equal(got.view(np.uint64), P.view(np.uint64)), (ta, tb)
            got, _ = M.emu_sgemm_ex(stored(A32, ta), stored(B32, tb), None, ta, tb)
            assert got.shape == P32.shape and np.array_equal(got.view(np.uint32), P32.view(np.uint32)), (ta, tb)


def pin_alpha_power_of_two(M):
    A = S.make("normal", 811, (9, 40), np.float64)
    B = S.make("normal", 812, (40, 8), np.float64)
    Cnan = np.full((9, 8), np.nan)
    P, _ = M.emu_dgemm(A, B, 10)
    P32, _ = M.emu_sgemm(A.astype(np.float32), B.astype(np.float32))
    for k in (3, -5):
        got, _ = M.emu_dgemm_ex(A, B, 10, Cnan, "N", "N", 2.0 ** k, 0.0)
        assert np.array_equal(got, np.ldexp(P, k)), k
        got, _ = M.emu_sgemm_ex(A.astype(np.float32), B.astype(np.float32), Cnan.astype(np.float32),
                                "N", "N", 2.0 ** k, 0.0)
        assert np.array_equal(got, np.ldexp(P32, k).astype(np.float32)), k


def _update_cases(rnd, eps_bits, want, n_cases=3, seed=5):
    """Seeded (alpha, P, beta, C) quadruples whose two-rounding update
    fl(fl(alpha P) + fl(beta C)) differs from both the fused form
    fl(alpha P + fl(beta C)) and the exact-sum form fl(alpha P + beta C).
    P is an integer product a b of small integers (exact in every emulated
    GEMM); beta C is chosen to cancel most of alpha P."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n_cases:
        a, b = (int(x) for x in rng.integers(100, 2 ** eps_bits, 2))
        P = Fraction(a * b)
        alpha = Fraction(float(want(rng.uniform(0.5, 2.0))))
        beta = Fraction(float(want(rng.uniform(0.5, 2.0))))
        C = Fraction(float(want(-float(alpha * P / beta) * (1 + rng.uniform(-2.0 ** -20, 2.0 ** -20)))))
        two = rnd(rnd(alpha * P) + rnd(beta * C))
        fused = rnd(alpha * P + rnd(beta * C))
        exact = rnd(alpha * P + beta * C)
        if two != fused and two != exact:
            out.append((a, b, alpha, beta, C, two))
    return out


def pin_update_rounding(M):
    # FP64: K = 1 integer operands |x| < 2^15 are captured exactly from nprod = 6 on
    for a, b, alpha, beta, C, two in _update_cases(to_f64, 15, np.float64):
        A = np.array([[float(a)]])
        B = np.array([[float(b)]])
        got, _ = M.emu_dgemm_ex(A, B, 6, np.array([[float(C)]]), "N", "N", float(alpha), float(beta))
        assert Fraction(float(got[0, 0])) == two, (a, b)
    # FP32: BF16-exact integers (|x| < 2^8) give an exact product
    for a, b, alpha, beta, C, two in _update_cases(to_f32, 8, np.float32):
        A = np.array([[a]], dtype=np.float32)
        B = np.array([[b]], dtype=np.float32)
        got, _ = M.emu_sgemm_ex(A, B, np.array([[float(C)]], dtype=np.float32), "N", "N",
                                float(alpha), float(beta))
        assert got.dtype == np.float32 and Fraction(float(got[0, 0])) == two, (a, b)


def pin_alpha_zero_and_k_zero(M):
    C0 = S.make("normal", 821, (6, 5), np.float64)
    Anan = np.full((6, 7), np.nan)
    Bnan = np.full((7, 5), np.nan)
    got, _ = M.emu_dgemm_ex(Anan, Bnan, 21, C0, "N", "N", 0.0, -2.0)
    assert np.array_equal(got, -2.0 * C0)
    got, _ = M.emu_dgemm_ex(Anan, Bnan, 21, np.full((6, 5), np.nan), "N", "N", 0.0, 0.0)
    assert got.shape == (6, 5) and not got.any()
    got, _ = M.emu_dgemm_ex(np.zeros((6, 0)), np.zeros((0, 5)), 6, C0, "N", "N", 1.0, 0.5)
    assert np.array_equal(got, 0.5 * C0)
    got, _ = M.emu_sgemm_ex(Anan.astype(np.float32), Bnan.astype(np.float32),
                            C0.astype(np.float32), "N", "N", 0.0, 3.0)
    assert np.array_equal(got, (np.float32(3.0) * C0.astype(np.float32)))
    # beta = 0: C is not read
    A = S.make("normal", 822, (6, 7), np.float64)
    B = S.make("normal", 823, (7, 5), np.float64)
    P, _ = M.emu_dgemm(A, B, 15)
    got, _ = M.emu_dgemm_ex(A, B, 15, np.full((6, 5), np.nan), "N", "N", 1.0, 0.0)
    assert np.array_equal(got, P)


PINS = [pin_transposes, pin_alpha_power_of_two, pin_update_rounding, pin_alpha_zero_and_k_zero]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_blas_composition(pin):
    pin(O)


def test_update_cases_exist():
    """The rounding pin is not vacuous: its cases separate the three forms."""
    assert len(_update_cases(to_f64, 15, np.float64)) == 3
    assert len(_update_cases(to_f32, 8, np.float32)) == 3


# ---------------------------------------------------------------------------
# Planted mistakes in the composition: each must be rejected by some pin.

SRC = os.path.join(os.path.dirname(O.__file__), "__init__.py")

MUTATIONS = {
    "fused_update": (
        "return (a * P + b * np.asarray(C, dtype=dtype)).astype(dtype)",
        "return (np.longdouble(a) * np.asarray(P, np.longdouble)"
        " + b * np.asarray(C, dtype=dtype)).astype(dtype)",
        [pin_update_rounding]),
    "alpha_applied_after_the_sum": (
        "return (a * P + b * np.asarray(C, dtype=dtype)).astype(dtype)",
        "return (a * (P + (b / a) * np.asarray(C, dtype=dtype))).astype(dtype)",
        [pin_update_rounding]),
    "transposes_ignored": (
        'return np.ascontiguousarray(X.T) if trans in ("T", "t", "C", "c") else X',
        "return X",
        [pin_transposes]),
    "beta_zero_reads_c": (
        "    if b == 0:\n        return (a * P).astype(dtype)\n",
        "",
        [pin_alpha_power_of_two, pin_alpha_zero_and_k_zero]),
    "alpha_zero_reads_operands": (
        "if alpha == 0 or opA.shape[1] == 0:",
        "if opA.shape[1] == 0:",
        [pin_alpha_zero_and_k_zero]),
}


def _mutant_module(text: str) -> types.ModuleType:
    """A copy of the oracle module built from modified source; it loads the
    same C library (its _HERE is the oracle directory)."""
    mod = types.ModuleType("oracle_blas_mutant")
    mod.__file__ = SRC
    exec(compile(text, SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_blas_mistake(name):
    old, new, pins = MUTATIONS[name]
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) >= 1, f"mutation site not found: {old[:50]}"
    M = _mutant_module(text.replace(old, new))
    pin_alpha_zero_and_k_zero(_mutant_module(text))      # the unmutated copy passes
    failures = []
    for pin in pins:
        try:
            pin(M)
        except (AssertionError, ValueError) as e:
            failures.append(repr(e)[:120])
    assert failures, f"no pin rejected the planted mistake '{name}'"
