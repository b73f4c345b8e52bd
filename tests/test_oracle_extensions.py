"""Pins of the oracle's two extensions of the scale-aware split (Sec. 9:
scale-aware decomposition and fallback handling; Sec. 4.3: inputs outside
the supported domain need a scaled or fallback extension).

K-binned scope (SCOPE_KBIN): the reduction is cut into groups of indices k
whose product terms have similar magnitude, each group is a row/column-scaled
emulated GEMM, and the groups are added in FP64.
  * the class of k from its definition, on hand-made operands;
  * integer operands whose every group product is exact: the groups add up to
    the exact product AB (no index lost or counted twice);
  * operands whose indices all share one class reduce to the row/column
    scope bit for bit;
  * K-direction scaling (1 % of B's rows 2^16 larger) reaches FP64-level
    error at nprod = 21, where the row/column scope does not.
Fallback (FALLBACK_FP64): a DGEMM whose status has any bit set is the plain
FP64 GEMM of its inputs instead.
  * in-domain inputs keep the emulation's bits, no fallback bit;
  * an entry below the BF16 range that meets a large entry of B: the exact
    product (which the emulation misses) and the fallback bit;
  * infinities: the IEEE pattern of a plain product.
"""
import os
import types
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import seeded_inputs as S


def pin_kbin_classes(M):
    # A: every column's largest entry 1 (after its row's scaling), B: rows at
    # 1, 2^-7, 2^-8, 2^-15, 2^-16, 2^-200 and a zero row, against a column
    # maximum of 1 (the first row): classes floor(-e / 8), e = ceil(log2) of
    # the row maxima, on both sides of every class boundary, the last capped
    A = np.ones((3, 7))
    B = np.zeros((7, 4))
    for k, e in enumerate([0, -7, -8, -15, -16, -200]):
        B[k, :] = 2.0 ** e
    cls = M.kbin_classes(A, B)
    assert list(cls) == [0, 0, 1, 1, 2, M.KBIN_MAX - 1, -1]


def pin_kbin_integers_exact(M):
    # |x| <= 2^7 integers (one or two slices, every group product exact), some
    # reduction rows of B 2^16 larger, one 2^-8 smaller: every exact output
    # needs at most 48 bits, so the FP64 sums of the groups are exact too
    rng = np.random.default_rng(3)
    A = rng.integers(-2 ** 7, 2 ** 7 + 1, (20, 300)).astype(np.float64)
    B = rng.integers(-2 ** 7, 2 ** 7 + 1, (300, 17)).astype(np.float64)
    B[::7] *= 2.0 ** 16                     # some reduction rows 2^16 larger
    B[5] *= 2.0 ** -8                       # one smaller
    A[:, 11] = 0.0                          # an index with a zero column (left out)
    assert len(set(M.kbin_classes(A, B)) - {-1}) >= 3
    C, st = M.emu_dgemm(A, B, 6, scope=M.SCOPE_KBIN)
    exact = [[sum(Fraction(float(A[m, k])) * Fraction(float(B[k, n])) for k in range(300))
              for n in range(17)] for m in range(20)]
    assert st == 0
    assert all(Fraction(float(C[m, n])) == exact[m][n] for m in range(20) for n in range(17))


def pin_kbin_single_class_is_rowcol(M):
    A = S.make("uniform", 81, (30, 520), np.float64)
    B = S.make("uniform", 82, (520, 20), np.float64)
    assert len(set(M.kbin_classes(A, B))) == 1
    for nprod in (6, 21):
        C1, _ = M.emu_dgemm(A, B, nprod, scope=M.SCOPE_KBIN)
        C2, _ = M.emu_dgemm(A, B, nprod, scope=M.SCOPE_ROWCOL)
        assert np.array_equal(C1.view(np.uint64), C2.view(np.uint64))


def pin_kbin_k_direction_accuracy(M):
    A = S.make("normal_scaled_rows", 83, (64, 2048), np.float64)
    B = S.make("normal_scaled_rows", 84, (2048, 64), np.float64)
    hi, lo = M.ref_gemm_dd(A, B)
    ab = np.abs(A) @ np.abs(B)

    def err(scope):
        C, st = M.emu_dgemm(A, B, 21, scope=scope)
        assert st == 0
        return float(np.max(np.abs((C - hi) - lo) / ab))
    e_kbin, e_rowcol = err(M.SCOPE_KBIN), err(M.SCOPE_ROWCOL)
    assert e_kbin < 2.0 ** -49 < e_rowcol, (e_kbin, e_rowcol)


def pin_fallback_in_domain(M):
    A = S.make("wide", 85, (40, 300), np.float64)
    B = S.make("uniform", 86, (300, 30), np.float64)
    C0 = S.make("normal", 87, (40, 30), np.float64)
    for nprod in (6, 21):
        P, st = M.emu_dgemm_ex(A, B, nprod, C0, alpha=1.5, beta=-0.5)
        F, stf = M.emu_dgemm_ex(A, B, nprod, C0, alpha=1.5, beta=-0.5, fallback=M.FALLBACK_FP64)
        assert st == stf == 0 and np.array_equal(P.view(np.uint64), F.view(np.uint64))


def pin_fallback_out_of_domain(M):
    rng = np.random.default_rng(5)
    A = rng.integers(-100, 101, (6, 9)).astype(np.float64)
    B = rng.integers(-100, 101, (9, 5)).astype(np.float64)
    A[:, 4] = 0.0
    A[2, 4] = 3.0 * 2.0 ** -140             # below Eq. (bf16rangefp64) and BF16 itself
    B[4, :] = 2.0 ** 127                    # meets a large entry: 3 2^-13 per output
    # (every exact output is an integer plus 0 or 3 2^-13: an FP64 value)
    exact = [[sum(Fraction(float(A[m, k])) * Fraction(float(B[k, n])) for k in range(9))
              for n in range(5)] for m in range(6)]
    P, st = M.emu_dgemm_ex(A, B, 21)
    assert st & M.ST_RANGE and not st & M.ST_FALLBACK
    assert Fraction(float(P[2, 0])) != exact[2][0]          # the emulation misses it
    F, stf = M.emu_dgemm_ex(A, B, 21, fallback=M.FALLBACK_FP64)
    assert stf & M.ST_RANGE and stf & M.ST_FALLBACK
    assert all(Fraction(float(F[m, n])) == exact[m][n] for m in range(6) for n in range(5))


def pin_fallback_infinity(M):
    A = S.make("normal", 88, (8, 12), np.float64)
    B = S.make("normal", 89, (12, 6), np.float64)
    A[1, 3] = np.inf
    B[7, 2] = -np.inf
    F, st = M.emu_dgemm_ex(A, B, 10, fallback=M.FALLBACK_FP64)
    want = A @ B
    assert st & M.ST_NAN and st & M.ST_FALLBACK
    assert np.array_equal(np.isnan(F), np.isnan(want)) and np.array_equal(np.isinf(F), np.isinf(want))
    fin = np.isfinite(want)
    assert np.allclose(F[fin], want[fin], rtol=1e-14, atol=0)


PINS = [pin_kbin_classes, pin_kbin_integers_exact, pin_kbin_single_class_is_rowcol,
        pin_kbin_k_direction_accuracy, pin_fallback_in_domain, pin_fallback_out_of_domain,
        pin_fallback_infinity]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_extension(pin):
    pin(O)


SRC = os.path.join(os.path.dirname(O.__file__), "__init__.py")

MUTATIONS = {
    "kbin_one_class": (
        "    cls = np.minimum((-e) // KBIN_WIDTH, KBIN_MAX - 1)",
        "    cls = np.zeros_like(e)",
        [pin_kbin_classes, pin_kbin_k_direction_accuracy]),
    "kbin_drops_first_class": (
        "        for b in range(KBIN_MAX):\n            ks = np.nonzero(cls == b)[0]\n            if ks.size == 0:\n                continue\n            Cb, sb",
        "        for b in range(1, KBIN_MAX):\n            ks = np.nonzero(cls == b)[0]\n            if ks.size == 0:\n                continue\n            Cb, sb",
        [pin_kbin_integers_exact]),
    "kbin_keeps_last_group_only": (
        "            C = Cb if first else Cb + C            # FP64, group order",
        "            C = Cb",
        [pin_kbin_integers_exact]),
    "kbin_width_off_by_one": (
        "    cls = np.minimum((-e) // KBIN_WIDTH, KBIN_MAX - 1)",
        "    cls = np.minimum((-e + 1) // KBIN_WIDTH, KBIN_MAX - 1)",
        [pin_kbin_classes]),
    "fallback_never_taken": (
        "    if fallback == FALLBACK_FP64 and st != 0:",
        "    if False:",
        [pin_fallback_out_of_domain, pin_fallback_infinity]),
    "fallback_always_taken": (
        "    if fallback == FALLBACK_FP64 and st != 0:",
        "    if fallback == FALLBACK_FP64:",
        [pin_fallback_in_domain]),
}


def _mutant_module(text: str) -> types.ModuleType:
    mod = types.ModuleType("oracle_ext_mutant")
    mod.__file__ = SRC
    exec(compile(text, SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_extension_mistake(name):
    old, new, pins = MUTATIONS[name]
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) >= 1, f"mutation site not found: {old[:50]}"
    M = _mutant_module(text.replace(old, new, 1))
    failures = []
    for pin in pins:
        try:
            pin(M)
        except (AssertionError, ValueError, IndexError) as e:
            failures.append(repr(e)[:120])
    assert failures, f"no pin rejected the planted mistake '{name}'"
