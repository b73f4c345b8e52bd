"""DGEMM parity at the shape boundaries where the library changes kernel or
grid, and at seeded random shapes over every product count.

The library picks, by shape, between the 32 x 32 x 16 kernel and the
16 x 16 x 32 kernel (64 x 64 or 128 x 64 tiles), and between one workgroup per
tile and a persistent grid (K <= 1024, more tiles than CUs, and for the
16 x 16 x 32 kernel an even number of k-blocks).  None of these choices may
change a bit of the result (Eq. fp64reconstruction with the executed order of
Sec. 6.3): sampled entries, corners included, are compared bit for bit with the
oracle.  Inputs are seeded and synthetic."""
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


def check_sampled(emu, M, N, K, nprod, seed, nsample=160):
    A = S.make("wide", seed, (M, K), np.float64)
    B = S.make("uniform", seed + 1, (K, N), np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    rng = np.random.default_rng(seed)
    r = np.concatenate([[0, M - 1, 0, M - 1], rng.integers(0, M, nsample)]).astype(np.int64)
    c = np.concatenate([[0, 0, N - 1, N - 1], rng.integers(0, N, nsample)]).astype(np.int64)
    ref, st = O.emu_dgemm_entries(A, B, r, c, nprod)
    assert st == 0
    got = np.ascontiguousarray(C[r, c])
    assert np.array_equal(got.view(np.uint64), ref.view(np.uint64)), (M, N, K, nprod)


# (M, N, K, nprod): both sides of each boundary
BOUNDARIES = [
    # K = 1024 is the last short reduction (32 k-blocks), 1025 the first long one
    (1100, 1100, 1024, 3), (1100, 1100, 1025, 3),
    (1100, 1100, 1024, 10), (1100, 1100, 1025, 10),
    (1100, 1100, 1024, 15), (1100, 1100, 1025, 15),
    (1100, 1100, 1024, 1), (1100, 1100, 1025, 1),
    # 256 tiles of 128 x 64 (d = 2, 3) or 256 x 64 (d = 1) is not "few"; 248 is
    (1024, 1984, 640, 6), (1024, 2048, 640, 6),
    (1024, 1984, 640, 3), (1024, 2048, 640, 3),
    (2048, 1984, 1100, 1), (2048, 2048, 1100, 1),
    # d = 6: exactly 256 tiles of 32 x 64 take one workgroup per tile, 272 a
    # persistent grid
    (512, 1024, 640, 21), (544, 1024, 640, 21),
    # odd k-block count with more tiles than CUs (the 16x16x32 kernel then
    # takes one tile per workgroup)
    (1040, 1100, 608, 21), (1040, 1100, 608, 36),
]


@pytest.mark.parametrize("M,N,K,nprod", BOUNDARIES)
def test_kernel_choice_boundaries_bit_exact(emu, M, N, K, nprod):
    check_sampled(emu, M, N, K, nprod, seed=7000 + M + N + K + nprod)


def _random_cases(n=20, seed=20260):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        M = int(rng.integers(1, 1400))
        N = int(rng.integers(1, 1400))
        K = int(rng.integers(1, 2300))
        nprod = int(rng.choice([1, 3, 6, 10, 15, 21, 26, 30, 33, 35, 36]))
        out.append((M, N, K, nprod))
    return out


@pytest.mark.parametrize("M,N,K,nprod", _random_cases())
def test_random_shapes_bit_exact(emu, M, N, K, nprod):
    check_sampled(emu, M, N, K, nprod, seed=9000 + M * 7 + N * 3 + K + nprod, nsample=96)


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (1, 700, 1300), (700, 1, 1300), (65, 3, 2049)])
@pytest.mark.parametrize("nprod", [1, 10, 21])
def test_degenerate_extents_bit_exact(emu, M, N, K, nprod):
    check_sampled(emu, M, N, K, nprod, seed=11000 + M + N + K + nprod, nsample=32)


def _random_forms(n=40, seed=31337):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        big = rng.random() < 0.3
        M = int(rng.integers(1, 2600 if big else 700))
        N = int(rng.integers(1, 2600 if big else 700))
        K = int(rng.integers(1, 2600))
        nprod = int(rng.choice([1, 3, 6, 10, 15, 21, 26, 30, 33, 35, 36]))
        out.append((M, N, K, nprod, str(rng.choice(["N", "T"])), str(rng.choice(["N", "T"])),
                    bool(rng.random() < 0.25)))
    return out


@pytest.mark.parametrize("M,N,K,nprod,ta,tb,rowcol", _random_forms())
def test_random_forms_and_scopes_bit_exact(emu, M, N, K, nprod, ta, tb, rowcol):
    """Seeded random shapes with transposed operands (op(A), op(B) of the BLAS
    form) and, for a quarter of them, the row/column exponent scope."""
    seed = 13000 + M + 3 * N + 7 * K + nprod
    A = S.make("wide", seed, (M, K), np.float64)
    B = S.make("normal", seed + 1, (K, N), np.float64)
    sA = np.ascontiguousarray(A.T) if ta == "T" else A
    sB = np.ascontiguousarray(B.T) if tb == "T" else B
    if rowcol:
        emu.set_split_scope(emu.SCOPE_ROWCOL)
    try:
        C = emu.dgemm_ex(dev(sA), dev(sB), nprod, None, ta, tb).cpu().numpy()
    finally:
        emu.set_split_scope(emu.SCOPE_OPERAND)
    rng = np.random.default_rng(seed)
    r = np.concatenate([[0, M - 1], rng.integers(0, M, 62)]).astype(np.int64)
    c = np.concatenate([[N - 1, 0], rng.integers(0, N, 62)]).astype(np.int64)
    ref, st = O.emu_dgemm_entries(A, B, r, c, nprod,
                                  scope=O.SCOPE_ROWCOL if rowcol else O.SCOPE_OPERAND)
    assert st == 0
    got = np.ascontiguousarray(C[r, c])
    assert np.array_equal(got.view(np.uint64), ref.view(np.uint64))


def _random_sgemm_forms(n=30, seed=4242):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        big = rng.random() < 0.3
        M = int(rng.integers(1, 2600 if big else 700))
        N = int(rng.integers(1, 2600 if big else 700))
        K = int(rng.integers(1, 3000))
        out.append((M, N, K, str(rng.choice(["N", "T"])), str(rng.choice(["N", "T"]))))
    return out


@pytest.mark.parametrize("M,N,K,ta,tb", _random_sgemm_forms())
def test_sgemm_random_forms_within_bounds(emu, M, N, K, ta, tb):
    """Emulated SGEMM at seeded random shapes (single pass and split-K, both
    operand orientations): every sampled entry within the per-entry bound of
    the omitted products plus the chunked FP32 accumulation, and the sample's
    normwise error within 4 K 2^-24, against a double-double reference."""
    import math
    seed = 17000 + M + 3 * N + 7 * K
    A = S.make("normal", seed, (M, K), np.float32)
    B = S.make("normal", seed + 1, (K, N), np.float32)
    sA = np.ascontiguousarray(A.T) if ta == "T" else A
    sB = np.ascontiguousarray(B.T) if tb == "T" else B
    C = emu.sgemm_ex(dev(sA), dev(sB), None, ta, tb).cpu().numpy()
    rng = np.random.default_rng(seed)
    r = np.concatenate([[0, M - 1], rng.integers(0, M, 94)]).astype(np.int64)
    c = np.concatenate([[N - 1, 0], rng.integers(0, N, 94)]).astype(np.int64)
    hi, lo = O.ref_dd_entries(A, B, r, c)
    ab = O.absprod_entries(A, B, r, c)
    got = np.ascontiguousarray(C[r, c]).astype(np.float64)
    err = np.abs((got - hi) - lo)
    esc_cap = 2.0 ** -22 + (6 * 256 + math.ceil(K / 256)) * 2.0 ** -24
    nz = ab > 0
    assert np.all(err[~nz] == 0.0)
    assert np.all(err[nz] <= esc_cap * ab[nz])
    if np.any(hi):
        assert np.sqrt(np.sum(err ** 2)) <= 4 * K * 2.0 ** -24 * np.sqrt(np.sum(hi ** 2))


# (M, N, K, tile rows, splits) the SGEMM picks: both tile heights, with and
# without split-K, ragged in every dimension
SGEMM_ROUTES = [
    (3001, 1999, 1111, 192, 1),
    (2990, 2100, 777, 128, 1),
    (1530, 1540, 1600, 192, 2),
    (1000, 900, 5000, 128, 4),
    (700, 600, 3000, 192, 12),
    (2048, 2048, 2048, 128, 1),
]


@pytest.mark.parametrize("M,N,K,tile,splits", SGEMM_ROUTES)
def test_sgemm_tile_routes_within_bounds(emu, M, N, K, tile, splits):
    """Each SGEMM configuration the shape can select (192- or 128-row tiles,
    one pass or split-K), checked like the random cases above."""
    import math
    seed = 19000 + M + N + K
    A = S.make("uniform", seed, (M, K), np.float32)
    B = S.make("normal", seed + 1, (K, N), np.float32)
    C = emu.sgemm(dev(A), dev(B)).cpu().numpy()
    rng = np.random.default_rng(seed)
    r = np.concatenate([[0, M - 1, M - 1, 0], rng.integers(0, M, 124)]).astype(np.int64)
    c = np.concatenate([[0, N - 1, 0, N - 1], rng.integers(0, N, 124)]).astype(np.int64)
    hi, lo = O.ref_dd_entries(A, B, r, c)
    ab = O.absprod_entries(A, B, r, c)
    err = np.abs((np.ascontiguousarray(C[r, c]).astype(np.float64) - hi) - lo)
    esc_cap = 2.0 ** -22 + (6 * 256 + math.ceil(K / 256)) * 2.0 ** -24
    assert np.all(err <= esc_cap * ab)
    assert np.sqrt(np.sum(err ** 2)) <= 4 * K * 2.0 ** -24 * np.sqrt(np.sum(hi ** 2))


def test_single_row_operands_with_numpy_strides(emu):
    """A (1, n) operand made from NumPy can carry a row stride of 1 (the
    stride of an extent-1 dimension is arbitrary); the binding accepts it and
    passes a leading dimension of n."""
    K, N = 1519, 1
    A = S.make("wide", 23001, (586, K), np.float64)
    B = S.make("uniform", 23002, (K, N), np.float64)
    Bt = np.ascontiguousarray(B.T)                 # shape (1, K), strides (8, 8)
    tB = torch.from_numpy(Bt).cuda()
    assert tB.shape == (1, K)
    C = emu.dgemm_ex(dev(A), tB, 3, None, "N", "T").cpu().numpy()
    ref, st = O.emu_dgemm(A, B, 3)
    assert st == 0 and np.array_equal(C.view(np.uint64), ref.view(np.uint64))
    row = torch.from_numpy(np.ascontiguousarray(S.make("normal", 23003, (K, 1), np.float32).T)).cuda()
    Cs = emu.sgemm(row, dev(S.make("normal", 23004, (K, 7), np.float32))).cpu().numpy()
    assert Cs.shape == (1, 7) and np.all(np.isfinite(Cs))
