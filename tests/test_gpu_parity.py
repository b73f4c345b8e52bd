"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars (from the exactness of the panel products, Sec. 4.3, and the omitted
products plus FP32 accumulation of the SGEMM, Sec. 4.2):
  * component planes, slices and exponents: bit-exact;
  * emulated DGEMM: bit-exact (every panel product is an exact FP32 value, so
    both sides add the same FP64 numbers in the same order);
  * emulated SGEMM: normwise error against an exact (FP64) reference at most
    twice the oracle's, below 4 K 2^-24, and a GEMM-scaled componentwise bound;
  * integer inputs whose products the retained set captures exactly: C = AB.
Inputs are seeded and synthetic (seeded_inputs); shapes span several tiles
with ragged tails.
"""
import math
import os

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
    E.lib()                                   # raises if libemu.so is missing
    return E


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def u16(t):
    return t.cpu().numpy().view(np.uint16)


def padded_view(a, extra=5):
    """Device copy of a with leading dimension cols + extra (ld > cols)."""
    R, C = a.shape
    big = np.zeros((R, C + extra), dtype=a.dtype)
    big[:, :C] = a
    return dev(big)[:, :C]


# ---------------------------------------------------------------------------
# split / pack


SPLIT_SHAPES = [(1, 1), (17, 255), (257, 33), (64, 300), (130, 1000)]


@pytest.mark.parametrize("as_b", [0, 1])
@pytest.mark.parametrize("shape", SPLIT_SHAPES)
@pytest.mark.parametrize("dist", ["normal", "wide"])
def test_split_f32_bit_exact(emu, shape, as_b, dist):
    X = S.make(dist, 101, shape, np.float32)
    emu.domain_status()
    ref, st = O.split_f32(X)
    got = u16(emu.split_f32(padded_view(X), as_b=bool(as_b)))
    assert np.array_equal(got, ref)
    assert emu.domain_status() == st


def test_split_f32_special_values_bit_exact(emu):
    vals = np.array([0.0, -0.0, 2.0 ** -103, -(2.0 ** -103) * 1.5, 1.0, -1.0 - 2.0 ** -23,
                     (2 - 2.0 ** -8) * 2.0 ** 127 * (1 - 2.0 ** -20), 3.0e38, 1.0 + 2.0 ** -8,
                     1.0 + 3 * 2.0 ** -8, 2.0 ** -126, 7.0e-39], dtype=np.float32)
    X = np.resize(vals, (8, 36)).astype(np.float32)
    emu.domain_status()
    ref, st = O.split_f32(X)
    got = u16(emu.split_f32(dev(X)))
    assert np.array_equal(got, ref)
    assert emu.domain_status() == st


def test_split_f32_domain_flags(emu):
    X = np.array([[np.nan, 1.0, 3.4e38, 1e-44]], dtype=np.float32)
    emu.domain_status()
    _, st = O.split_f32(X)
    emu.split_f32(dev(X))
    got = emu.domain_status()
    assert got == st and got & emu.STATUS_NAN and got & emu.STATUS_OVERFLOW
    assert got & emu.STATUS_SUBNORMAL


def _f64_cases():
    rng = np.random.default_rng(7)
    ints = rng.integers(-2 ** 15, 2 ** 15 + 1, (40, 70)).astype(np.float64)
    single = np.zeros((33, 65))
    single[5, 7] = 1.0 / 3.0
    # magnitude classes 22 bits apart with 7-bit mantissas: each level's
    # maximum comes from the next class, so the speculated chain (9 bits per
    # level) is wrong at every level and every pass replays
    cls = rng.integers(0, 6, (45, 66))
    mant = 1.0 + rng.integers(0, 128, (45, 66)) / 128.0
    sign = np.where(rng.integers(0, 2, (45, 66)) == 1, -1.0, 1.0)
    classes = sign * mant * np.exp2(-22.0 * cls)
    return {
        "replay_every_level": classes,
        "uniform": S.make("uniform", 201, (130, 257), np.float64),
        "normal": S.make("normal", 202, (33, 70), np.float64),
        "wide": S.make("wide", 203, (70, 129), np.float64),
        "integers": ints,                      # v drops faster than 9 bits: replays
        "zero": np.zeros((17, 40)),
        "single": single,
        "scaled_rows": S.make("normal_scaled_rows", 204, (200, 64), np.float64),
    }


@pytest.mark.parametrize("mode", [O.SPLIT_SYM, O.SPLIT_LITERAL])
@pytest.mark.parametrize("as_b", [0, 1])
@pytest.mark.parametrize("case", list(_f64_cases().keys()))
def test_split_f64_bit_exact(emu, case, as_b, mode):
    X = _f64_cases()[case]
    emu.domain_status()
    ref, v, _, st = O.split_f64(X, mode)
    emu.set_split_mode(mode)
    try:
        s, vg = emu.split_f64(padded_view(X), as_b=bool(as_b))
        got = u16(s)
        vg = vg.cpu().numpy()
    finally:
        emu.set_split_mode(emu.SPLIT_SYM)
    assert np.array_equal(vg, v), (vg, v)
    assert np.array_equal(got, ref)
    assert emu.domain_status() == st


@pytest.mark.parametrize("nprod", [6, 21])
def test_dgemm_replay_every_level_bit_exact(emu, nprod):
    """(Deeper products of these classes fall below the FP32 range.)"""
    X = _f64_cases()["replay_every_level"]
    _, v, _, _ = O.split_f64(X)
    assert all(v[r + 1] < v[r] - 9 for r in range(5))        # every level mis-speculated
    A, B = X[:, :60], np.ascontiguousarray(X[:, 6:66].T)    # 45 x 60 and 60 x 45
    ref, st = O.emu_dgemm(A, B, nprod)
    C = emu.dgemm(dev(A), dev(np.ascontiguousarray(B)), nprod).cpu().numpy()
    assert st == 0 and np.array_equal(C.view(np.uint64), ref.view(np.uint64))


def test_split_f64_domain_flags(emu):
    for X in (np.array([[1.0, 2.0 ** -130]]), np.array([[2.0 ** 200, 1.0]]),
              np.array([[2.0 ** -120 * (1 + 2.0 ** -30), 2.0 ** -121]])):
        emu.domain_status()
        _, _, _, st = O.split_f64(X)
        emu.split_f64(dev(X))
        assert emu.domain_status() == st
    # NaN/Inf lie outside every domain the paper defines and the slices are
    # unspecified; only the NaN/Inf bit is required of both sides.
    X = np.array([[1.0, np.inf], [np.nan, 2.0]])
    emu.domain_status()
    _, _, _, st = O.split_f64(X)
    emu.split_f64(dev(X))
    assert st & O.ST_NAN and emu.domain_status() & emu.STATUS_NAN


# ---------------------------------------------------------------------------
# emulated DGEMM: bit-exact


GEMM_SHAPES = [(1, 1, 1), (33, 17, 40), (130, 70, 600), (257, 129, 513), (64, 192, 256)]


@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
@pytest.mark.parametrize("dist", ["uniform", "wide"])
def test_dgemm_bit_exact(emu, shape, nprod, dist):
    M, N, K = shape
    A = S.make(dist, 301, (M, K), np.float64)
    B = S.make(dist, 302, (K, N), np.float64)
    ref, st = O.emu_dgemm(A, B, nprod)
    C = emu.dgemm(padded_view(A), padded_view(B), nprod).cpu().numpy()
    assert st == 0
    assert np.array_equal(C.view(np.uint64), ref.view(np.uint64)), \
        f"{np.count_nonzero(C != ref)} of {C.size} differ, max |d| {np.max(np.abs(C - ref))}"


@pytest.mark.parametrize("nprod", [6, 21])
def test_dgemm_ld_and_output_stride(emu, nprod):
    M, N, K = 70, 90, 300
    A = S.make("normal", 311, (M, K), np.float64)
    B = S.make("normal", 312, (K, N), np.float64)
    ref, _ = O.emu_dgemm(A, B, nprod)
    Cbig = torch.full((M, N + 7), 7.0, dtype=torch.float64, device="cuda")
    emu.dgemm(padded_view(A, 3), padded_view(B, 9), nprod, C=Cbig[:, :N])
    out = Cbig.cpu().numpy()
    assert np.array_equal(out[:, :N], ref)
    assert np.all(out[:, N:] == 7.0)                  # nothing written past N


@pytest.mark.parametrize("nprod", [6, 10, 15, 21])
def test_dgemm_integers_exact(emu, nprod):
    rng = np.random.default_rng(8)
    A = rng.integers(-2 ** 15, 2 ** 15 + 1, (65, 700)).astype(np.float64)
    B = rng.integers(-2 ** 15, 2 ** 15 + 1, (700, 66)).astype(np.float64)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    assert np.array_equal(C.astype(np.int64), A.astype(np.int64) @ B.astype(np.int64))


def test_dgemm_panel_sum_at_fp32_limit(emu):
    """Slice entries of magnitude 256 units over a full panel: the panel sum
    reaches 2^24 units, the FP32 limit of exactness."""
    K = 512
    A = np.full((64, K), 1.0)
    B = np.full((K, 64), -1.0)
    A[::3, ::5] = 255.0 / 256.0
    ref, _ = O.emu_dgemm(A, B, 21)
    C = emu.dgemm(dev(A), dev(B), 21).cpu().numpy()
    assert np.array_equal(C, ref)


def test_dgemm_literal_mode_bit_exact(emu):
    A = S.make("uniform", 321, (100, 300), np.float64)
    B = S.make("uniform", 322, (300, 80), np.float64)
    ref, _ = O.emu_dgemm(A, B, 15, mode=O.SPLIT_LITERAL)
    emu.set_split_mode(emu.SPLIT_LITERAL)
    try:
        C = emu.dgemm(dev(A), dev(B), 15).cpu().numpy()
    finally:
        emu.set_split_mode(emu.SPLIT_SYM)
    assert np.array_equal(C, ref)


# ---------------------------------------------------------------------------
# emulated SGEMM: tolerance


def sgemm_bounds(K):
    return 4 * K * 2.0 ** -24, 2.0 ** -22 + (6 * 256 + math.ceil(K / 256)) * 2.0 ** -24


def check_sgemm(emu, A, B, Cg=None):
    M, K = A.shape
    Corc, _ = O.emu_sgemm(A, B)
    if Cg is None:
        Cg = emu.sgemm(padded_view(A), padded_view(B)).cpu().numpy()
    ref = O.ref_gemm_f64(A, B)
    ab = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    e_orc = O.e_F(Corc, ref) if np.any(ref) else 0.0
    e_gpu = O.e_F(Cg, ref) if np.any(ref) else 0.0
    esc, zero_abs = O.e_scaled(Cg, ref, ab)
    ef_cap, esc_cap = sgemm_bounds(K)
    assert e_gpu <= 2 * e_orc + 1e-12, (e_gpu, e_orc)
    assert e_gpu <= ef_cap
    assert esc <= esc_cap and zero_abs == 0.0
    return e_gpu, e_orc


@pytest.mark.parametrize("shape", GEMM_SHAPES + [(256, 256, 256)])
@pytest.mark.parametrize("dist", ["uniform", "normal"])
def test_sgemm_tolerance(emu, shape, dist):
    M, N, K = shape
    A = S.make(dist, 401, (M, K), np.float32)
    B = S.make(dist, 402, (K, N), np.float32)
    check_sgemm(emu, A, B)


def test_sgemm_scaled_rows_tolerance(emu):
    A = S.make("normal_scaled_rows", 411, (200, 1500), np.float32)
    B = S.make("normal_scaled_rows", 412, (1500, 150), np.float32)
    check_sgemm(emu, A, B)


def test_sgemm_integer_pins(emu):
    rng = np.random.default_rng(9)
    A = rng.integers(-256, 257, (70, 256)).astype(np.float32)
    B = rng.integers(-256, 257, (256, 90)).astype(np.float32)
    C = emu.sgemm(dev(A), dev(B)).cpu().numpy()
    assert np.array_equal(C.astype(np.int64), A.astype(np.int64) @ B.astype(np.int64))
    A = rng.integers(-1000, 1001, (70, 16)).astype(np.float32)
    B = rng.integers(-1000, 1001, (16, 90)).astype(np.float32)
    C = emu.sgemm(dev(A), dev(B)).cpu().numpy()
    assert np.array_equal(C.astype(np.int64), A.astype(np.int64) @ B.astype(np.int64))


def test_sgemm_identity(emu):
    A = S.make("normal", 421, (100, 300), np.float32)
    C = emu.sgemm(dev(A), dev(np.eye(300, dtype=np.float32))).cpu().numpy()
    assert np.array_equal(C, A)


def test_sgemm_deterministic(emu):
    A = dev(S.make("normal", 431, (300, 700), np.float32))
    B = dev(S.make("normal", 432, (700, 250), np.float32))
    c1 = emu.sgemm(A, B).cpu().numpy()
    c2 = emu.sgemm(A, B).cpu().numpy()
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))


# ---------------------------------------------------------------------------
# boundary behaviour on the device


def test_k_zero_writes_zero(emu):
    C = torch.full((5, 7), 3.0, device="cuda")
    emu.sgemm(torch.empty((5, 0), device="cuda"), torch.empty((0, 7), device="cuda"), C=C)
    assert torch.all(C == 0).item()
    C = torch.full((5, 7), 3.0, dtype=torch.float64, device="cuda")
    emu.dgemm(torch.empty((5, 0), dtype=torch.float64, device="cuda"),
              torch.empty((0, 7), dtype=torch.float64, device="cuda"), 6, C=C)
    assert torch.all(C == 0).item()


def test_dgemm_domain_status(emu):
    A = np.ones((4, 4))
    A[0, 0] = 2.0 ** -130
    emu.domain_status()
    emu.dgemm(dev(A), dev(np.ones((4, 4))), 6)
    assert emu.domain_status() & emu.STATUS_RANGE
    emu.dgemm(dev(np.ones((4, 4))), dev(np.ones((4, 4))), 6)
    assert emu.domain_status() == 0


def test_dgemm_inexact_status_for_tiny_operands(emu):
    """Operands of magnitude 2^-45 are inside Eq. (bf16rangefp64) and their
    six slices are normal BF16 values, yet the lower panel products of
    nprod = 21 fall below FP32's normal range (unit 2^(vA_i + vB_j - 16) down
    to 2^-151): the library reports EMU_STATUS_INEXACT, and the oracle, which
    rounds each exact panel sum to FP32, finds inexact panels there.  At
    nprod = 6 every unit is at least 2^-124: no flag, and the result is the
    unscaled operands' result times 2^-90 bit for bit (powers of two commute
    with every rounding of the method while nothing leaves the normal range)."""
    A = S.make("uniform", 361, (70, 600), np.float64)
    B = S.make("uniform", 362, (600, 50), np.float64)
    As, Bs = np.ldexp(A, -45), np.ldexp(B, -45)
    emu.domain_status()
    C6 = emu.dgemm(dev(As), dev(Bs), 6).cpu().numpy()
    assert emu.domain_status() == 0
    ref6, st6 = O.emu_dgemm(As, Bs, 6)
    assert st6 == 0 and np.array_equal(C6, ref6)
    assert np.array_equal(C6, np.ldexp(emu.dgemm(dev(A), dev(B), 6).cpu().numpy(), -90))
    emu.dgemm(dev(As), dev(Bs), 21)
    assert emu.domain_status() == emu.STATUS_INEXACT
    _, st21 = O.emu_dgemm(As, Bs, 21)
    assert st21 == O.ST_INEXACT32


def test_dgemm_inexact_status_for_fp32_overflow(emu):
    """Operands near 2^64: the leading panel product's bound 2^(vA_0 + vB_0 + 8)
    exceeds FP32's range, so the status is raised; the split itself is exact."""
    A = np.ldexp(S.make("uniform", 363, (40, 300), np.float64), 64)
    B = np.ldexp(S.make("uniform", 364, (300, 30), np.float64), 64)
    emu.domain_status()
    emu.dgemm(dev(A), dev(B), 6)
    assert emu.domain_status() == emu.STATUS_INEXACT


def test_workspace_limit_gives_enomem(emu):
    emu.release_workspace()
    os.environ["EMU_WORKSPACE_LIMIT"] = "4096"
    try:
        with pytest.raises(emu.EmuError) as ei:
            emu.sgemm(dev(np.ones((300, 300), np.float32)), dev(np.ones((300, 300), np.float32)))
        assert ei.value.code == emu.EMU_ENOMEM
    finally:
        del os.environ["EMU_WORKSPACE_LIMIT"]
    C = emu.sgemm(dev(np.ones((30, 30), np.float32)), dev(np.ones((30, 30), np.float32)))
    assert torch.all(C == 30).item()


# ---------------------------------------------------------------------------
# degenerate operands of the method


@pytest.mark.parametrize("nprod", [6, 21])
def test_dgemm_zero_and_single_entry_operands(emu, nprod):
    """A = 0 gives all-zero slices (the zero-residual rule) and C = 0; a single
    nonzero entry gives its exact slices; both bit-exact with the oracle."""
    B = S.make("wide", 341, (300, 70), np.float64)
    A = np.zeros((90, 300))
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    assert not C.any()
    A[17, 123] = -3.0e-5
    ref, _ = O.emu_dgemm(A, B, nprod)
    C = emu.dgemm(dev(A), dev(B), nprod).cpu().numpy()
    assert np.array_equal(C, ref)


@pytest.mark.parametrize("shape", [(1, 300, 5000), (300, 1, 5000), (1, 1, 70000)])
def test_vector_shapes(emu, shape):
    """GEMV-like shapes and a long single dot product (many panels)."""
    M, N, K = shape
    A = S.make("wide", 351, (M, K), np.float64)
    B = S.make("uniform", 352, (K, N), np.float64)
    ref, _ = O.emu_dgemm(A, B, 10)
    assert np.array_equal(emu.dgemm(dev(A), dev(B), 10).cpu().numpy(), ref)
    A32, B32 = A.astype(np.float32), B.astype(np.float32)
    if M * N >= 64:
        check_sgemm(emu, A32, B32)
    else:
        # one output number: the ratio to the oracle's error is a single sample
        # (here about 2x either way), so only the absolute bounds of R5 apply
        Cg = emu.sgemm(dev(A32), dev(B32)).cpu().numpy()
        ref64 = O.ref_gemm_f64(A32, B32)
        esc, _ = O.e_scaled(Cg, ref64, np.abs(A32.astype(np.float64)) @ np.abs(B32.astype(np.float64)))
        ef_cap, esc_cap = sgemm_bounds(K)
        assert O.e_F(Cg, ref64) <= ef_cap and esc <= esc_cap
