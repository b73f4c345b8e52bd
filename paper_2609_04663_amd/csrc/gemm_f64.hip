// Emulated DGEMM: the N_p(d) retained component products of the fixed
// six-slice split (Eq. fp64productcounts), each evaluated per reduction panel
// of 256 on bf16 MFMA with FP32 accumulation, then widened and added in FP64
// (Eq. fp64reconstruction, Algorithm fp64, Sec. 6.3) -- the FP64
// widen-and-accumulate epilogue is fused into the k-loop.
//
// Exactness of a panel product.  With operand-wide exponents every entry of
// slice A_i is an integer multiple of 2^(vA_i - 8) of magnitude <= 2^vA_i, so a
// panel sum of 256 slice products is an integer multiple of
// 2^(vA_i + vB_j - 16) below 2^24 such units: every partial sum is an FP32
// value and the MFMA accumulation is exact in any order.  The FP64 result then
// depends only on the order of the FP64 additions, which here is the paper's:
// panel ascending, diagonal l = i + j ascending, i ascending inside a diagonal.
//
// Workgroup: 4 waves in a 2 x 2 grid; wave tile (32 BM) x 32, output tile
// (64 BM) x 64.  Per k-block of 32 the d planes of both operands are copied
// straight into LDS (global_load_lds_dwordx4), double-buffered.  Each wave
// keeps one FP32 accumulator set per product for the whole panel (all N_p
// live, so every fragment read from LDS feeds every product that uses it) and
// an FP64 accumulator tile.
#include "gemm_common.h"

namespace emu {
namespace {

template <int D, int BM>
struct Cfg {
    static constexpr int P = D * (D + 1) / 2;
    static constexpr int MT = 64 * BM, NT = DGEMM_NT;
    static constexpr int A_BYTES = MT * 64, B_BYTES = NT * 64;
    static constexpr int STAGE = D * (A_BYTES + B_BYTES);
    static constexpr int A_PARTS = A_BYTES / 1024, B_PARTS = B_BYTES / 1024;
    static constexpr int CHUNKS = D * (A_PARTS + B_PARTS);
    static_assert(CHUNKS % 4 == 0, "chunks must split evenly over 4 waves");
    static_assert(2 * STAGE <= 160 * 1024, "LDS");
};

template <int D, int BM>
__global__ __launch_bounds__(256, 1) void gemm_f64_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, double *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc, int nt_m, int nt_n) {
    using K = Cfg<D, BM>;
    __shared__ __attribute__((aligned(1024))) char stage0[K::STAGE];
    __shared__ __attribute__((aligned(1024))) char stage1[K::STAGE];

    int tm, tn;
    tile_coords<8>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * K::MT, n0 = (int64_t)tn * K::NT;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = (int64_t)KB * RpadA * 64;
    const int64_t b_plane = (int64_t)KB * RpadB * 64;

    auto issue = [&](int kb, char *base) {
#pragma unroll 1
        for (int i = 0; i < K::CHUNKS / 4; ++i) {
            const int ch = wave + 4 * i;
            if (ch < D * K::A_PARTS) {
                const int c = ch / K::A_PARTS, part = ch % K::A_PARTS;
                const char *src = Ag + c * a_plane + ((int64_t)kb * RpadA + m0) * 64 + part * 1024;
                copy_1k(src, base + c * K::A_BYTES + part * 1024, lane);
            } else {
                const int cc = ch - D * K::A_PARTS;
                const int c = cc / K::B_PARTS, part = cc % K::B_PARTS;
                const char *src = Bg + c * b_plane + ((int64_t)kb * RpadB + n0) * 64 + part * 1024;
                copy_1k(src, base + D * K::A_BYTES + c * K::B_BYTES + part * 1024, lane);
            }
        }
    };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);

    // One 16-index sub-step on the stage at `base`: every retained product.
    // first: the panel's first sub-step, whose MFMAs start from zero (no
    // separate zeroing of the accumulators, so no second live set).
    auto substep = [&](const char *base, int off, f32x16 (&acc)[K::P][BM], bool first) {
        const char *At = base + (wm * 32 * BM) * 64;
        const char *Bt = base + D * K::A_BYTES + (wn * 32) * 64;
        bf16x8 af[D][BM], bf[D];
#pragma unroll
        for (int c = 0; c < D; ++c) {
            bf[c] = lds_frag(Bt + c * K::B_BYTES, off);
#pragma unroll
            for (int b = 0; b < BM; ++b) af[c][b] = lds_frag(At + c * K::A_BYTES + b * 32 * 64, off);
        }
        // product q = l (l + 1) / 2 + i is A_i B_(l - i): diagonal l ascending,
        // i ascending (all indices are compile-time constants after unrolling)
#pragma unroll
        for (int l = 0; l < D; ++l)
#pragma unroll
            for (int i = 0; i <= l; ++i)
#pragma unroll
                for (int b = 0; b < BM; ++b)
                    acc[l * (l + 1) / 2 + i][b] =
                        mfma(af[i][b], bf[l - i], first ? f32x16{} : acc[l * (l + 1) / 2 + i][b]);
    };

    double acc64[BM][16];
#pragma unroll
    for (int b = 0; b < BM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc64[b][r] = 0.0;

    // Outer loop: reduction panels of 256; inner loop: double-buffered k-blocks
    // (same schedule as the FP32 kernel).  After each panel every product is
    // widened exactly and added in FP64, in the executed order.
    issue(0, stage0);
    int kb = 0;
    for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
        const int p1 = min(KB, p0 + KB_PER_PANEL);
        f32x16 acc[K::P][BM];
        {   // first k-block of the panel (peeled: its first sub-step starts from zero)
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            char *cur = (kb & 1) ? stage1 : stage0;
            char *nxt = (kb & 1) ? stage0 : stage1;
            if (kb + 1 < KB) issue(kb + 1, nxt);
            substep(cur, off0, acc, true);
            substep(cur, off1, acc, false);
            ++kb;
        }
        for (; kb < p1; ++kb) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            char *cur = (kb & 1) ? stage1 : stage0;
            char *nxt = (kb & 1) ? stage0 : stage1;
            if (kb + 1 < KB) issue(kb + 1, nxt);
            substep(cur, off0, acc, false);
            substep(cur, off1, acc, false);
        }
#pragma unroll
        for (int q = 0; q < K::P; ++q)
#pragma unroll
            for (int b = 0; b < BM; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc64[b][r] += (double)acc[q][b][r];
    }

#pragma unroll
    for (int b = 0; b < BM; ++b) {
        const int64_t col = n0 + wn * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = m0 + wm * 32 * BM + b * 32 + acc_row(lane, r);
            if (row < M && col < N) C[row * ldc + col] = acc64[b][r];
        }
    }
}

template <int D, int BM>
hipError_t launch_t(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M, int64_t N,
                    int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, hipStream_t s) {
    using K = Cfg<D, BM>;
    const int nt_m = (int)((M + K::MT - 1) / K::MT), nt_n = (int)((N + K::NT - 1) / K::NT);
    gemm_f64_kernel<D, BM><<<nt_m * nt_n, 256, 0, s>>>(Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc,
                                                       nt_m, nt_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f64(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M,
                           int64_t N, int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
                           int d, hipStream_t s) {
    switch (d) {
        case 3: return launch_t<3, 2>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, s);
        case 4: return launch_t<4, 1>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, s);
        case 5: return launch_t<5, 1>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, s);
        case 6: return launch_t<6, 1>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace emu
