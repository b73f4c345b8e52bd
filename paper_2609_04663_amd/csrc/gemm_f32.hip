// Emulated SGEMM: the six retained component products of Eq. (fp32six),
// Sec. 4.2, on bf16 MFMA (v_mfma_f32_32x32x16_bf16) with FP32 accumulation.
//
// Workgroup: 256 threads = 4 waves in a 2 x 2 grid, output tile 192 x 128,
// wave tile 96 x 64 (3 x 2 MFMA blocks of 32 x 32).  Per k-block of 32
// reduction indices the three BF16 planes of both operands (3 x 12 KB of A,
// 3 x 8 KB of B) are copied straight from the packed buffers into LDS with
// global_load_lds_dwordx4, double-buffered, so the copy of k-block kb + 1
// overlaps the MFMAs of k-block kb.  Each wave reads every fragment once per
// 16-index sub-step and issues all six products on it: B fragments of the three
// planes stay in registers while the A planes are walked (A0: B0, B1, B2;
// A1: B0, B1; A2: B0), 36 MFMAs per sub-step on 15 fragments.  The wave tile
// is sized so that the three accumulator sets below (288 registers) leave the
// register allocator room: 128 x 64 spills.
//
// Accumulation: A0B0 goes to one FP32 accumulator set, the five smaller
// products to another; at the end of every reduction panel of 256 (the
// paper's B_K, Sec. 6.1/6.3) the two are combined and added into an FP32 block
// total.  Keeping the leading product apart stops the small products from
// being rounded against the large partial sums inside the MFMA accumulator.
#include "gemm_common.h"

namespace emu {
namespace {

constexpr int MT = SGEMM_MT, NT = SGEMM_NT, NC = 3, RB = MT / 64;
constexpr int A_BYTES = MT * 64;                    // one plane, one k-block
constexpr int B_BYTES = NT * 64;
constexpr int STAGE = NC * (A_BYTES + B_BYTES);     // 72 KB
constexpr int A_CHUNKS = NC * A_BYTES / 1024;       // 36
constexpr int B_CHUNKS = NC * B_BYTES / 1024;       // 24

__global__ __launch_bounds__(256, 1) void gemm_f32_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, float *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc, int nt_m, int nt_n) {
    __shared__ __attribute__((aligned(1024))) char stage0[STAGE];
    __shared__ __attribute__((aligned(1024))) char stage1[STAGE];

    int tm, tn;
    tile_coords<4>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * MT, n0 = (int64_t)tn * NT;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = (int64_t)KB * RpadA * 64;
    const int64_t b_plane = (int64_t)KB * RpadB * 64;

    // Copy issue: a runtime loop keeps the per-chunk addresses out of registers.
    auto issue = [&](int kb, char *base) {
#pragma unroll 1
        for (int i = 0; i < A_CHUNKS / 4; ++i) {
            const int ch = wave * (A_CHUNKS / 4) + i;
            const int c = ch / (A_BYTES / 1024), part = ch % (A_BYTES / 1024);
            const char *src = Ag + c * a_plane + ((int64_t)kb * RpadA + m0) * 64 + part * 1024;
            copy_1k(src, base + c * A_BYTES + part * 1024, lane);
        }
#pragma unroll 1
        for (int i = 0; i < B_CHUNKS / 4; ++i) {
            const int ch = wave * (B_CHUNKS / 4) + i;
            const int c = ch / (B_BYTES / 1024), part = ch % (B_BYTES / 1024);
            const char *src = Bg + c * b_plane + ((int64_t)kb * RpadB + n0) * 64 + part * 1024;
            copy_1k(src, base + NC * A_BYTES + c * B_BYTES + part * 1024, lane);
        }
    };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);

    // One 16-index sub-step on the stage at `base`: 36 MFMAs into hi / lo.
    auto substep = [&](const char *base, int off, f32x16 (&hi)[RB][2], f32x16 (&lo)[RB][2]) {
        const char *At = base + (wm * 32 * RB) * 64;
        const char *Bt = base + NC * A_BYTES + (wn * 64) * 64;
        bf16x8 bfr[NC][2];
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) bfr[c][cb] = lds_frag(Bt + c * B_BYTES + cb * 32 * 64, off);
        bf16x8 afr[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) afr[rb] = lds_frag(At + rb * 32 * 64, off);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) hi[rb][cb] = mfma(afr[rb], bfr[0][cb], hi[rb][cb]);
#pragma unroll
        for (int j = 1; j < 3; ++j)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) lo[rb][cb] = mfma(afr[rb], bfr[j][cb], lo[rb][cb]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) afr[rb] = lds_frag(At + A_BYTES + rb * 32 * 64, off);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) lo[rb][cb] = mfma(afr[rb], bfr[j][cb], lo[rb][cb]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) afr[rb] = lds_frag(At + 2 * A_BYTES + rb * 32 * 64, off);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) lo[rb][cb] = mfma(afr[rb], bfr[0][cb], lo[rb][cb]);
    };

    f32x16 blk[RB][2];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) blk[i][j] = f32x16{};

    // Outer loop: reduction panels of 256 (the FP32 reconstruction unit).
    // Inner loop: k-blocks of 32, double-buffered; at the top of trip kb the copy
    // of k-block kb has landed (own copies: vmcnt; other waves': barrier) and
    // every wave has finished reading the other stage, which the copy of
    // k-block kb + 1 then refills.
    issue(0, stage0);
    int kb = 0;
    for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
        const int p1 = min(KB, p0 + KB_PER_PANEL);
        f32x16 hi[RB][2], lo[RB][2];
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                hi[i][j] = f32x16{};
                lo[i][j] = f32x16{};
            }
        for (; kb < p1; ++kb) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            char *cur = (kb & 1) ? stage1 : stage0;
            char *nxt = (kb & 1) ? stage0 : stage1;
            if (kb + 1 < KB) issue(kb + 1, nxt);
            substep(cur, off0, hi, lo);
            substep(cur, off1, hi, lo);
        }
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) blk[i][j] += lo[i][j] + hi[i][j];
    }

    // Store the wave tile.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int64_t col = n0 + wn * 64 + cb * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 32 * RB + rb * 32 + acc_row(lane, r);
                if (row < M && col < N) C[row * ldc + col] = blk[rb][cb][r];
            }
        }
}

}  // namespace

hipError_t launch_gemm_f32(const uint16_t *Ap, const uint16_t *Bp, float *C, int64_t M, int64_t N,
                           int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, hipStream_t s) {
    const int nt_m = (int)((M + MT - 1) / MT), nt_n = (int)((N + NT - 1) / NT);
    gemm_f32_kernel<<<nt_m * nt_n, 256, 0, s>>>(Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, nt_m,
                                               nt_n);
    return hipGetLastError();
}

}  // namespace emu
