"""GPU parity of the K-binned scale-aware scope (EMU_SCOPE_KBIN).

The scale-aware decomposition (Sec. 9) extended along the reduction: the
indices k are classed by the magnitude of their product terms, every class is
a row/column-scaled emulated DGEMM of its own columns of op(A) and rows of
op(B), and the class products are added in FP64 in ascending class order.
Expected values are the oracle's form of the same scope:

  * bit-exact outputs and equal status words on ragged shapes, every nprod,
    the four transposition forms with alpha and beta;
  * integer operands with K-direction scaling: the exact product;
  * operands whose indices share one class: the row/column scope bit for bit;
  * reduction rows 2^300 larger than the rest (far beyond what row and column
    weights can cover): no status bit and FP64-level error on the outputs the
    small rows alone make;
  * the armed fallback still replaces a call that raised a bit;
  * the rectangular workloads with 1 % of the rows scaled by 2^16 at their
    full sizes: sampled entries bit-exact against the oracle, and the error
    against the double-double reference well below the row/column scope's,
    at FP64 level for nprod = 21.
"""
import numpy as np
import pytest
import torch

import oracle as O
import seeded_inputs as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kbin():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    E.set_split_scope(E.SCOPE_KBIN)
    yield E
    E.set_split_scope(E.SCOPE_OPERAND)
    E.set_fallback(E.FALLBACK_NONE)
    E.release_workspace()
    torch.cuda.empty_cache()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def stored(X, trans):
    return np.ascontiguousarray(X.T) if trans == "T" else X


def bits_equal(a, b):
    return np.array_equal(np.asarray(a).view(np.uint64), np.asarray(b).view(np.uint64))


@pytest.mark.parametrize("shape", [(130, 90, 700), (257, 129, 1500), (5, 3, 11)])
@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
def test_kbin_bit_exact(kbin, shape, nprod):
    M, N, K = shape
    A = S.make("normal_scaled_rows", 1401, (M, K), np.float64)
    B = S.make("normal_scaled_rows", 1402, (K, N), np.float64)
    assert len(set(O.kbin_classes(A, B)) - {-1}) >= 2 or K < 100
    kbin.domain_status()
    got = kbin.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    st = kbin.domain_status()
    ref, sto = O.emu_dgemm(A, B, nprod, scope=O.SCOPE_KBIN)
    assert st == sto == 0
    assert bits_equal(got, ref)


@pytest.mark.parametrize("ta,tb", [("N", "N"), ("T", "N"), ("N", "T"), ("T", "T")])
@pytest.mark.parametrize("alpha,beta", [(-1.25, 0.5), (1.0, 0.0), (3.0, 0.0)])
def test_kbin_blas_forms(kbin, ta, tb, alpha, beta):
    M, N, K = 97, 66, 515
    A = S.make("normal_scaled_rows", 1403, (M, K), np.float64)
    B = S.make("normal_scaled_rows", 1404, (K, N), np.float64)
    B[::9] *= 2.0 ** -20                   # a third, smaller class along k
    C0 = S.make("normal", 1405, (M, N), np.float64)
    if beta == 0.0:
        C0[0, 0] = np.nan                  # beta = 0: C is not read
    got = kbin.dgemm_ex(dev(stored(A, ta)), dev(stored(B, tb)), 15, dev(C0.copy()), ta, tb, alpha,
                        beta).cpu().numpy()
    ref, st = O.emu_dgemm_ex(stored(A, ta), stored(B, tb), 15, C0, ta, tb, alpha, beta,
                             scope=O.SCOPE_KBIN)
    assert st == 0 and kbin.domain_status() == 0
    assert bits_equal(got, ref)


def test_kbin_integers_exact(kbin):
    """|x| <= 2^7 integers, every 7th reduction row of B 2^16 larger and one
    2^-8 smaller, one zero column of A: the exact product (every output needs
    at most 51 bits, so the FP64 sums of the groups are exact)."""
    rng = np.random.default_rng(1406)
    M, N, K = 200, 150, 3000
    A = rng.integers(-2 ** 7, 2 ** 7 + 1, (M, K)).astype(np.float64)
    B = rng.integers(-2 ** 7, 2 ** 7 + 1, (K, N)).astype(np.float64)
    B[::7] *= 2.0 ** 16
    B[5] *= 2.0 ** -8
    A[:, 11] = 0.0
    assert len(set(O.kbin_classes(A, B)) - {-1}) >= 3
    exact = A.astype(np.int64) @ np.rint(B * 2.0 ** 8).astype(np.int64)
    got = kbin.dgemm(dev(A), dev(B), 6).cpu().numpy()
    assert kbin.domain_status() == 0
    assert np.array_equal(np.rint(got * 2.0 ** 8).astype(np.int64), exact)
    assert np.array_equal(got * 2.0 ** 8, np.rint(got * 2.0 ** 8))


def test_kbin_single_class_is_rowcol(kbin):
    A = S.make("uniform", 1407, (150, 800), np.float64)
    B = S.make("uniform", 1408, (800, 70), np.float64)
    assert len(set(O.kbin_classes(A, B))) == 1
    for nprod in (6, 21):
        got = kbin.dgemm(dev(A), dev(B), nprod).cpu().numpy()
        kbin.set_split_scope(kbin.SCOPE_ROWCOL)
        try:
            rc = kbin.dgemm(dev(A), dev(B), nprod).cpu().numpy()
        finally:
            kbin.set_split_scope(kbin.SCOPE_KBIN)
        assert bits_equal(got, rc)


def test_kbin_reduction_rows_2p300(kbin):
    """1 % of B's rows 2^300 larger; half of A's rows miss them (zero in
    those columns), so their outputs come from the small rows alone.  Row and
    column weights cannot hold both (the small rows sit 2^300 below their
    column maximum: ROWCOL flags range); the K-binned scope puts them in
    groups of their own."""
    M, N, K = 128, 96, 2048
    A = S.make("normal", 1409, (M, K), np.float64)
    B = S.make("normal", 1410, (K, N), np.float64)
    big = S.permutation(1411, K)[:K // 100]
    B[big] *= 2.0 ** 300
    A[: M // 2, big] = 0.0
    kbin.domain_status()
    got = kbin.dgemm(dev(A), dev(B), 21).cpu().numpy()
    assert kbin.domain_status() == 0
    ref, st = O.emu_dgemm(A, B, 21, scope=O.SCOPE_KBIN)
    assert st == 0 and bits_equal(got, ref)
    hi, _ = O.ref_gemm_dd(A, B)
    for part in (slice(0, M // 2), slice(M // 2, M)):
        e = O.e_F(got[part], hi[part])
        print(f"rows {part}: e_F {e:.3e}", flush=True)
        assert e < 2.0 ** -49
    kbin.set_split_scope(kbin.SCOPE_ROWCOL)
    try:
        kbin.dgemm(dev(A), dev(B), 21)
        assert kbin.domain_status() & kbin.STATUS_RANGE
    finally:
        kbin.set_split_scope(kbin.SCOPE_KBIN)


@pytest.mark.parametrize("ab", [(1.0, 0.0), (-0.5, 2.0)])
def test_kbin_with_the_fallback(kbin, ab):
    """An entry below BF16's range meeting a row of B at 2^127 stays out of the
    domain in every scope: the armed fallback gives the exact product."""
    alpha, beta = ab
    rng = np.random.default_rng(1412)
    M, N, K = 70, 50, 400
    A = rng.integers(-100, 101, (M, K)).astype(np.float64)
    B = rng.integers(-100, 101, (K, N)).astype(np.float64)
    k = K // 2
    A[:, k] = 0.0
    A[M // 3, k] = 3.0 * 2.0 ** -140
    B[k, :] = 2.0 ** 127
    C0 = rng.integers(-100, 101, (M, N)).astype(np.float64)
    kbin.set_fallback(kbin.FALLBACK_FP64)
    try:
        kbin.domain_status()
        got = kbin.dgemm_ex(dev(A), dev(B), 21, dev(C0.copy()), "N", "N", alpha, beta).cpu().numpy()
        st = kbin.domain_status()
    finally:
        kbin.set_fallback(kbin.FALLBACK_NONE)
    assert st & kbin.STATUS_FALLBACK
    ref, sto = O.emu_dgemm_ex(A, B, 21, C0, "N", "N", alpha, beta, scope=O.SCOPE_KBIN,
                              fallback=O.FALLBACK_FP64)
    assert sto & O.ST_FALLBACK
    assert bits_equal(got, ref)


def test_kbin_in_domain_fallback_keeps_the_emulation(kbin):
    A = S.make("normal_scaled_rows", 1413, (120, 600), np.float64)
    B = S.make("normal_scaled_rows", 1414, (600, 80), np.float64)
    kbin.set_fallback(kbin.FALLBACK_FP64)
    try:
        kbin.domain_status()
        got = kbin.dgemm(dev(A), dev(B), 10).cpu().numpy()
        st = kbin.domain_status()
    finally:
        kbin.set_fallback(kbin.FALLBACK_NONE)
    ref, sto = O.emu_dgemm_ex(A, B, 10, scope=O.SCOPE_KBIN, fallback=O.FALLBACK_FP64)
    assert st == sto == 0 and bits_equal(got, ref)


@pytest.mark.parametrize("shape", [(16384, 16384, 512), (1024, 1024, 65536)])
def test_kbin_rectangular_scaled_rows(kbin, shape):
    """The rectangular workloads with 1 % of the rows of A and of B scaled by
    2^16, at full size: 192 sampled entries bit-exact against the oracle; the
    sampled error against the double-double reference is well below the
    row/column scope's at nprod 10 and 21, and at FP64 level (below 2^-49)
    at nprod 21."""
    M, N, K = shape
    sa, sb = S.seeds(5)
    A = S.make("normal_scaled_rows", sa, (M, K), np.float64)
    B = S.make("normal_scaled_rows", sb, (K, N), np.float64)
    rng = np.random.default_rng(M + K + 1)
    rows = rng.integers(0, M, 192)
    cols = rng.integers(0, N, 192)
    dA, dB = dev(A), dev(B)
    r_t, c_t = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    hi, _ = O.ref_dd_entries(A, B, rows, cols)
    for nprod in (10, 21):
        print(f"kbin {shape} nprod={nprod}", flush=True)
        C = kbin.dgemm(dA, dB, nprod)
        got = C[r_t, c_t].cpu().numpy()
        del C
        assert kbin.domain_status() == 0
        ref, st = O.emu_dgemm_entries(A, B, rows, cols, nprod, scope=O.SCOPE_KBIN)
        assert st == 0 and bits_equal(got, ref)
        kbin.set_split_scope(kbin.SCOPE_ROWCOL)
        try:
            C = kbin.dgemm(dA, dB, nprod)
            got_rc = C[r_t, c_t].cpu().numpy()
            del C
        finally:
            kbin.set_split_scope(kbin.SCOPE_KBIN)
        e_kb, e_rc = O.e_F(got, hi), O.e_F(got_rc, hi)
        print(f"{shape} nprod={nprod}: e_F kbin {e_kb:.3e} rowcol {e_rc:.3e}", flush=True)
        assert e_kb < e_rc / 4
        if nprod == 21:
            assert e_kb < 2.0 ** -49
    del dA, dB
    kbin.release_workspace()
    torch.cuda.empty_cache()
