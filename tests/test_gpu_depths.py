"""GPU parity at every depth of the triangular product selection,
Eq. (product-selection): nprod = N_p(d) for d = 1, 2 (one or three products)
and d = 7 .. 11 (26 .. 36 products, the 16 x 16 x 32 MFMA kernel), and the
choice between the two DGEMM kernels that depths 1 .. 5 make by shape.  The bar is the same as for the paper's depths:
bit-exact against the oracle (every panel product is an exact FP32 value and
both sides add them in the same FP64 order).  Inputs are seeded and synthetic;
the shapes span several tiles of every kernel with ragged tails."""
import numpy as np
import pytest
import torch

import oracle as O
import seeded_inputs as S

pytestmark = pytest.mark.gpu

NEW = [1, 3, 26, 30, 33, 35, 36]
SHAPES = [(1, 1, 1), (33, 17, 40), (130, 70, 600), (257, 129, 513)]


@pytest.fixture(scope="module")
def emu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    return E


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def padded_view(a, extra=5):
    R, C = a.shape
    big = np.zeros((R, C + extra), dtype=a.dtype)
    big[:, :C] = a
    return dev(big)[:, :C]


def same_bits(got, ref):
    return np.array_equal(got.view(np.uint64), ref.view(np.uint64))


@pytest.mark.parametrize("nprod", NEW)
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dist", ["uniform", "wide"])
def test_dgemm_depths_bit_exact(emu, shape, nprod, dist):
    M, N, K = shape
    A = S.make(dist, 901, (M, K), np.float64)
    B = S.make(dist, 902, (K, N), np.float64)
    ref, st = O.emu_dgemm(A, B, nprod)
    assert st == 0
    C = emu.dgemm(padded_view(A), padded_view(B), nprod).cpu().numpy()
    assert same_bits(C, ref), \
        f"{np.count_nonzero(C != ref)} of {C.size} differ, max |d| {np.max(np.abs(C - ref))}"


@pytest.mark.parametrize("d", range(1, 12))
def test_structured_operands_closed_form(emu, d):
    """The K = 1 operands whose slices are fixed by hand (a = 1 + 2^-9 + ... +
    2^-36, x = 2^-60): each depth gives a different closed-form result."""
    nprod = sum(1 for i in range(6) for j in range(6) if i + j < d)
    a = sum(2.0 ** (-9 * i) for i in range(5))
    x = 2.0 ** -60
    A = np.array([[a], [x]])
    B = np.array([[a, x]])
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    c00 = sum(sum(1 for i in range(5) if 0 <= l - i <= 4) * 2.0 ** (-9 * l)
              for l in range(min(d, 6)))
    c10 = sum(x * 2.0 ** (-9 * j) for j in range(5) if 5 + j < d)
    assert C[0, 0] == c00 and C[1, 0] == c10 and C[0, 1] == c10
    assert C[1, 1] == (x * x if d == 11 else 0.0)


@pytest.mark.parametrize("nprod", [1, 36])
def test_dgemm_depths_ld_and_output_stride(emu, nprod):
    M, N, K = 70, 90, 300
    A = S.make("normal", 911, (M, K), np.float64)
    B = S.make("normal", 912, (K, N), np.float64)
    ref, _ = O.emu_dgemm(A, B, nprod)
    Cbig = torch.full((M, N + 7), 7.0, dtype=torch.float64, device="cuda")
    emu.dgemm(padded_view(A, 3), padded_view(B, 9), nprod, C=Cbig[:, :N])
    out = Cbig.cpu().numpy()
    assert same_bits(np.ascontiguousarray(out[:, :N]), ref)
    assert np.all(out[:, N:] == 7.0)


@pytest.mark.parametrize("nprod", [3, 36])
def test_dgemm_integers_exact_from_depth_3(emu, nprod):
    """Integers below 2^15 in magnitude occupy two slices, so every depth from
    3 on captures their products exactly."""
    rng = np.random.default_rng(9)
    A = rng.integers(-2 ** 15, 2 ** 15 + 1, (65, 700)).astype(np.float64)
    B = rng.integers(-2 ** 15, 2 ** 15 + 1, (700, 66)).astype(np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    exact = A.astype(np.int64) @ B.astype(np.int64)
    if nprod >= 6:
        assert np.array_equal(C.astype(np.int64), exact)
    else:
        ref, _ = O.emu_dgemm(A, B, nprod)
        assert same_bits(C, ref)


@pytest.mark.parametrize("ta,tb", [("N", "N"), ("T", "T")])
@pytest.mark.parametrize("nprod", [1, 36])
def test_dgemm_ex_depths_bit_exact(emu, ta, tb, nprod):
    M, N, K = 130, 70, 600
    A = S.make("wide", 921, (M, K), np.float64)
    B = S.make("uniform", 922, (K, N), np.float64)
    C0 = S.make("normal", 923, (M, N), np.float64)
    sA = np.ascontiguousarray(A.T) if ta == "T" else A
    sB = np.ascontiguousarray(B.T) if tb == "T" else B
    for alpha, beta in ((1.0, 0.0), (-2.5, 0.75)):
        ref, _ = O.emu_dgemm_ex(sA, sB, nprod, C0, ta, tb, alpha, beta)
        got = emu.dgemm_ex(dev(sA), dev(sB), nprod, dev(C0.copy()), ta, tb, alpha,
                           beta).cpu().numpy()
        assert same_bits(got, ref), (alpha, beta)


@pytest.mark.parametrize("nprod", [1, 36])
def test_dgemm_rowcol_depths_bit_exact(emu, nprod):
    M, N, K = 257, 129, 513
    A = S.make("normal_scaled_rows", 931, (M, K), np.float64)
    B = S.make("wide", 932, (K, N), np.float64)
    ref, st = O.emu_dgemm(A, B, nprod, scope=O.SCOPE_ROWCOL)
    emu.set_split_scope(emu.SCOPE_ROWCOL)
    try:
        C = emu.dgemm(padded_view(A), padded_view(B), nprod).cpu().numpy()
    finally:
        emu.set_split_scope(emu.SCOPE_OPERAND)
    assert same_bits(C, ref)


@pytest.mark.parametrize("K", [640, 600])
@pytest.mark.parametrize("nprod", [10, 15, 21, 36])
def test_dgemm_persistent_tiles_bit_exact(emu, K, nprod):
    """More output tiles than CUs and a short reduction: both DGEMM kernels run
    persistent workgroups that walk several tiles each, the copy ring running
    on across tile boundaries.  The 16 x 16 x 32 kernel (nprod 21, 36) needs an
    even k-block count (K = 640) and takes one tile per workgroup otherwise
    (K = 600); the 32 x 32 x 16 kernel (nprod 10, 15 at these short
    reductions: 324 tiles of 64 x 64) takes either.  Sampled entries,
    including the last tile row and column."""
    M = N = 1100
    A = S.make("wide", 961, (M, K), np.float64)
    B = S.make("uniform", 962, (K, N), np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    rng = np.random.default_rng(K + nprod)
    r = np.concatenate([[0, M - 1, 0, M - 1, M - 5], rng.integers(0, M, 379)]).astype(np.int64)
    c = np.concatenate([[0, 0, N - 1, N - 1, N - 7], rng.integers(0, N, 379)]).astype(np.int64)
    ref, st = O.emu_dgemm_entries(A, B, r, c, nprod)
    assert st == 0
    assert same_bits(np.ascontiguousarray(C[r, c]), ref)


@pytest.mark.parametrize("nprod", [1, 3, 6])
def test_dgemm_persistent_large_tiles_bit_exact(emu, nprod):
    """The persistent 32 x 32 x 16 kernel with its larger tiles (256 x 64 for nprod 1,
    128 x 64 for 3 and 6): 2100 x 2100 outputs give more tiles than CUs."""
    M = N = 2100
    K = 640
    A = S.make("normal", 971, (M, K), np.float64)
    B = S.make("wide", 972, (K, N), np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    rng = np.random.default_rng(nprod)
    r = np.concatenate([[0, M - 1, 0, M - 1], rng.integers(0, M, 380)]).astype(np.int64)
    c = np.concatenate([[0, 0, N - 1, N - 1], rng.integers(0, N, 380)]).astype(np.int64)
    ref, st = O.emu_dgemm_entries(A, B, r, c, nprod)
    assert st == 0
    assert same_bits(np.ascontiguousarray(C[r, c]), ref)


# (M, N, K, nprod, kernel the shape selects).  "32x32": the 32 x 32 x 16
# kernel; "wide": the 16 x 16 x 32 kernel with 64 x 64 tiles; "wide128": the
# same with 128 x 64 tiles; "persistent": its persistent grid (more 64 x 64
# tiles than CUs, an even number of k-blocks of 32, K <= 1024).  Depths 1 and
# 3 take the wide kernel when their 256- or 128-row tiles number fewer than
# 256; depths 1 and 2 also for K > 1024 (depth 1 then on 128 x 64 tiles);
# depths 4 and 5 only for K > 1024.
ROUTES = [
    (2100, 1900, 1500, 1, "wide128"),     # 270 tiles of 256 x 64, 47 k-blocks
    (2100, 1900, 640, 1, "32x32"),        # the same grid, short reduction
    (1000, 1000, 1100, 1, "wide"),        # 64 tiles of 256 x 64, 35 k-blocks
    (1500, 1000, 640, 3, "persistent"),   # 192 tiles of 128 x 64 -> 384 of 64 x 64
    (700, 600, 1100, 3, "wide"),          # long reduction
    (2100, 1900, 1500, 6, "32x32"),       # 510 tiles of 128 x 64
    (1000, 900, 1100, 6, "wide"),         # 120 tiles of 128 x 64
    (1500, 1000, 640, 6, "persistent"),
    (700, 600, 1100, 10, "wide"),         # long reduction, odd k-block count
    (700, 600, 1000, 10, "32x32"),
    (700, 600, 1100, 15, "wide"),
    (700, 600, 1000, 15, "32x32"),        # K <= 1024
]


@pytest.mark.parametrize("M,N,K,nprod,kernel", ROUTES)
def test_dgemm_kernel_routes_bit_exact(emu, M, N, K, nprod, kernel):
    """Each kernel that depths 1 .. 5 can select, at ragged shapes: sampled
    entries, including the corners of the last tile row and column, are
    bit-identical to the oracle's."""
    A = S.make("wide", 981 + nprod, (M, K), np.float64)
    B = S.make("normal", 982 + nprod, (K, N), np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    rng = np.random.default_rng(M + K + nprod)
    r = np.concatenate([[0, M - 1, 0, M - 1, M - 3], rng.integers(0, M, 251)]).astype(np.int64)
    c = np.concatenate([[0, 0, N - 1, N - 1, N - 5], rng.integers(0, N, 251)]).astype(np.int64)
    ref, st = O.emu_dgemm_entries(A, B, r, c, nprod)
    assert st == 0
    assert same_bits(np.ascontiguousarray(C[r, c]), ref)
