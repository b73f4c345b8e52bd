// Emulated SGEMM: the six retained component products of Eq. (fp32six),
// Sec. 4.2, on bf16 MFMA (v_mfma_f32_32x32x16_bf16) with FP32 accumulation.
//
// Workgroup: 256 threads = 4 waves in a 2 x 2 grid, output tile 192 x 128,
// wave tile 96 x 64 (3 x 2 MFMA blocks of 32 x 32); a 128 x 128 tile (wave
// 64 x 64) serves grids whose 192-row tiles would leave CUs idle.  Per k-block
// of 32 reduction indices the three BF16 planes of both operands (3 x 12 KB of
// A, 3 x 8 KB of B) are copied straight from the packed buffers into LDS with
// global_load_lds_dwordx4, double-buffered, so the copy of k-block kb + 1
// overlaps the MFMAs of k-block kb.  Each wave reads every fragment once per
// 16-index sub-step and issues all six products on it: B fragments of the three
// planes stay in registers while the A planes are walked (A0: B0, B1, B2;
// A1: B0, B1; A2: B0), 36 MFMAs per sub-step on 15 fragments.  The wave tile
// is sized so that the three accumulator sets below (288 registers) leave the
// register allocator room: 128 x 64 spills.
//
// Accumulation: A0B0 goes to one FP32 accumulator set (hi), flushed into an
// FP32 block total at the end of every reduction panel of 256 (the paper's
// B_K, Sec. 6.1/6.3); the five smaller products go to another set (lo) that
// runs over the whole reduction and is added to the block total at the end.
// Keeping the leading product apart stops the small products from being
// rounded against the large partial sums; lo itself is about 2^-8 of C, so
// its own rounding over the full length stays far below FP32 level, and the
// panel flush reads only hi (half the accumulator reads of flushing both).
#include "gemm_common.h"

namespace emu {
namespace {

constexpr int NT = SGEMM_NT, NC = 3;

// RB 32-row blocks per wave: output tile (64 RB) x 128, wave tile (32 RB) x 64.
template <int RB>
__global__ __launch_bounds__(256, 1) void gemm_f32_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, float *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc, float alpha,
    float beta, int nt_m, int nt_n, int kb_per_split, float *__restrict__ part) {
    constexpr int MT = 64 * RB;
    constexpr int A_BYTES = MT * 64;                    // one plane, one k-block
    constexpr int B_BYTES = NT * 64;
    constexpr int STAGE = NC * (A_BYTES + B_BYTES);     // 60 KB (RB = 3), 48 KB (RB = 2)
    __shared__ __attribute__((aligned(1024))) char stage0[STAGE];
    __shared__ __attribute__((aligned(1024))) char stage1[STAGE];

    int tm, tn;
    tile_coords<4>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const unsigned lane16 = (unsigned)lane * 16u;   // copy offset of this lane
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * MT, n0 = (int64_t)tn * NT;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = plane_elems(KB, RpadA) * 2;
    const int64_t b_plane = plane_elems(KB, RpadB) * 2;

    // Copy issue for one k-block: wave w moves 1 KB parts [RB w, RB w + RB) of
    // each A plane and [2w, 2w + 2) of each B plane, so every address is a
    // wave-uniform base plus a compile-time offset.  Copy j < 3 RB is A plane
    // j / RB, part j % RB; copy 3 RB + j is B plane j / 2, part j % 2.
    static_assert(A_BYTES / 1024 == 4 * RB && B_BYTES / 1024 == 8, "part split");
    constexpr int AC = NC * RB, COPIES = AC + 6;
    const int64_t a_base = m0 * 64 + wave * RB * 1024;
    const int64_t b_base = n0 * 64 + wave * 2 * 1024;
    auto issue_one = [&](int kb, char *base, auto j_c) {
        constexpr int j = decltype(j_c)::value;
        if constexpr (j < AC)
            copy_1k(Ag + (int64_t)kb * RpadA * 64 + a_base + (j / RB) * a_plane + (j % RB) * 1024,
                    base + wave * RB * 1024 + (j / RB) * A_BYTES + (j % RB) * 1024, lane16);
        else
            copy_1k(Bg + (int64_t)kb * RpadB * 64 + b_base + ((j - AC) / 2) * b_plane +
                        ((j - AC) % 2) * 1024,
                    base + NC * A_BYTES + wave * 2 * 1024 + ((j - AC) / 2) * B_BYTES +
                        ((j - AC) % 2) * 1024,
                    lane16);
    };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);

    // Operand fragments of one 16-index sub-step: the three B planes (2 column
    // blocks) and the three A planes (RB row blocks).  One register set: each
    // fragment is re-read for the next sub-step right after its last use in the
    // current one, except B0, whose last use is the sub-step's last MFMA: it has
    // a second buffer (b0 below) that is filled at the start of the sub-step.
    struct Frags {
        bf16x8 b[NC][2];
        bf16x8 a[NC][RB];
    };
    const int at0 = (wm * 32 * RB) * 64, bt0 = NC * A_BYTES + (wn * 64) * 64;
    auto read_a = [&](const char *base, int off, int c, int rb) {
        return lds_frag(base + at0 + c * A_BYTES + rb * 32 * 64, off);
    };
    auto read_b = [&](const char *base, int off, int c, int cb) {
        return lds_frag(base + bt0 + c * B_BYTES + cb * 32 * 64, off);
    };
    // One sub-step in 12 RB slots.  MFMA t is product g = t / G (G = 2 RB) of
    // (A0B0 | A0B1 A0B2 A1B0 A1B1 A2B0) on block (rb, cb) = ((t % G) / 2, t % 2):
    // A0B0 goes to hi, the five smaller products to lo, product-major so that
    // consecutive MFMAs never share an accumulator.  After MFMA t come the reads
    // of the next sub-step (stage nbase, lane offset noff) of the fragments whose
    // last use was MFMA t, then copy t / 2 of k-block ckb (even t, t / 2 < NCOPY).
    // Latency cover of every read: at least 4 RB MFMAs.
    // zero: the panel's first sub-step (hi starts at 0); zero_lo: the first
    // sub-step of the whole reduction (lo starts at 0).
    constexpr int PI[6] = {0, 0, 0, 1, 1, 2}, PJ[6] = {0, 1, 2, 0, 1, 0};
    auto step = [&](Frags &f, const bf16x8 (&b0)[2], bf16x8 (&b0n)[2], f32x16 (&hi)[RB][2],
                    f32x16 (&lo)[RB][2], auto zero_c, auto zero_lo_c, const char *nbase, int noff,
                    int ckb, char *cdst, auto ncopy_c) {
        constexpr bool zero = decltype(zero_c)::value;
        constexpr bool zero_lo = decltype(zero_lo_c)::value;
        constexpr int NCOPY = decltype(ncopy_c)::value;
        constexpr int G = 2 * RB;
        static_for<12 * RB>([&](auto t_c) {
            constexpr int t = decltype(t_c)::value;
            constexpr int g = t / G, rb = (t % G) / 2, cb = t % 2;
            constexpr int i = PI[g], j = PJ[g];
            const bf16x8 &bop = (j == 0) ? b0[cb] : f.b[j][cb];
            if constexpr (g == 0)
                hi[rb][cb] = mfma(f.a[0][rb], bop, zero ? f32x16{} : hi[rb][cb]);
            else
                lo[rb][cb] = mfma(f.a[i][rb], bop, (zero_lo && g == 1) ? f32x16{} : lo[rb][cb]);
            order_fence();
            // last uses: B0 -> second buffer at t = 0, 1; A0[r] at 2G + 1 + 2r;
            // B2[c] at 3G - 2 + c; A1[r] at 4G + 1 + 2r; B1[c] at 5G - 2 + c;
            // A2[r] at 5G + 1 + 2r (RB = 3: 13 + 2r, 16 + c, 25 + 2r, 28 + c, 31 + 2r)
            constexpr int ua0 = t - (2 * G + 1), ua1 = t - (4 * G + 1), ua2 = t - (5 * G + 1);
            constexpr int ub2 = t - (3 * G - 2), ub1 = t - (5 * G - 2);
            if constexpr (t < 2) b0n[t] = read_b(nbase, noff, 0, t);
            if constexpr (ua0 >= 0 && ua0 % 2 == 0 && ua0 / 2 < RB) f.a[0][ua0 / 2] = read_a(nbase, noff, 0, ua0 / 2);
            if constexpr (ub2 == 0 || ub2 == 1) f.b[2][ub2] = read_b(nbase, noff, 2, ub2);
            if constexpr (ua1 >= 0 && ua1 % 2 == 0 && ua1 / 2 < RB) f.a[1][ua1 / 2] = read_a(nbase, noff, 1, ua1 / 2);
            if constexpr (ub1 == 0 || ub1 == 1) f.b[1][ub1] = read_b(nbase, noff, 1, ub1);
            if constexpr (ua2 >= 0 && ua2 % 2 == 0 && ua2 / 2 < RB) f.a[2][ua2 / 2] = read_a(nbase, noff, 2, ua2 / 2);
            order_fence();
            if constexpr (t % 2 == 0 && t / 2 < NCOPY)
                issue_one(ckb, cdst, std::integral_constant<int, t / 2>{});
            order_fence();
        });
    };

    f32x16 blk[RB][2];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) blk[i][j] = f32x16{};

    // Software pipeline over k-blocks (two LDS stages).  Entering trip kb the
    // sub-step-0 fragments of kb are in registers and the copy of kb + 1 is in
    // flight.  The trip (1) reads the sub-step-1 fragments of kb while the
    // sub-step-0 MFMAs run; (2) waits for its own copies of kb + 1 and its LDS
    // reads, then barriers: now every wave is done reading stage kb and every
    // copy of kb + 1 has landed; (3) starts the copy of kb + 2 into stage kb and
    // reads the sub-step-0 fragments of kb + 1 while the sub-step-1 MFMAs run.
    // The copy past the last k-block re-reads the last one (in bounds, unused).
    // split-K: this workgroup reduces k-blocks [kb_lo, kb_hi), whole panels
    const int kb_lo = blockIdx.y * kb_per_split;
    const int kb_hi = min(KB, kb_lo + kb_per_split);
    static_for<COPIES>([&](auto j_c) { issue_one(kb_lo, stage0, j_c); });
    static_for<COPIES>([&](auto j_c) { issue_one(min(kb_lo + 1, kb_hi - 1), stage1, j_c); });
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(COPIES) : "memory");
    __syncthreads();
    Frags f;
    bf16x8 b0a[2], b0b[2];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) f.b[c][cb] = read_b(stage0, off0, c, cb);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) f.a[c][rb] = read_a(stage0, off0, c, rb);
    }
    b0a[0] = f.b[0][0];
    b0a[1] = f.b[0][1];
    int kb = kb_lo;
    f32x16 lo[RB][2];
    for (int p0 = kb_lo; p0 < kb_hi; p0 += KB_PER_PANEL) {
        const int p1 = min(kb_hi, p0 + KB_PER_PANEL);
        f32x16 hi[RB][2];
        auto kblock = [&](auto first_c, auto first_lo_c) {
            char *cur = (kb & 1) ? stage1 : stage0;
            char *nxt = (kb & 1) ? stage0 : stage1;
            step(f, b0a, b0b, hi, lo, first_c, first_lo_c, cur, off1, 0, cur,
                 std::integral_constant<int, 0>{});
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            pipeline_barrier();
            step(f, b0b, b0a, hi, lo, std::false_type{}, std::false_type{}, nxt, off0,
                 min(kb + 2, kb_hi - 1), cur, std::integral_constant<int, COPIES>{});
            __builtin_amdgcn_sched_barrier(0);
        };
        if (p0 == kb_lo) kblock(std::true_type{}, std::true_type{});
        else kblock(std::true_type{}, std::false_type{});
        for (++kb; kb < p1; ++kb) kblock(std::false_type{}, std::false_type{});
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) blk[i][j] += hi[i][j];
    }
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) blk[i][j] += lo[i][j];
    // the last trips issued (unused) copies: let them land before the workgroup
    // ends and its LDS is handed to another workgroup
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // Store the wave tile.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int64_t col = n0 + wn * 64 + cb * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 32 * RB + rb * 32 + acc_row(lane, r);
                if (row < M && col < N) {
                    if (part != nullptr)   // split-K: this split's sum, added by reduce_splits
                        part[((int64_t)blockIdx.y * M + row) * N + col] = blk[rb][cb][r];
                    else
                        C[row * ldc + col] = out_update(blk[rb][cb][r], alpha, beta, C + row * ldc + col);
                }
            }
        }
}

// ---------------------------------------------------------------------------
// Streamed split (the alternative of Sec. 6.2 in which the components are made
// where they are consumed): the same products, accumulation and tile walk as
// gemm_f32_kernel, but the workgroup reads op(A) and op(B) in FP32 and splits
// each k-block into its three BF16 planes itself (Eq. fp32split, the split
// kernel's arithmetic), writing them to LDS in the packed layout, so no packed
// planes go through HBM.  Each element is split once per workgroup that reads
// it.  The FP32 k-block kb + 2 is loaded into registers during k-block kb,
// split and written into the stage that k-block kb has just released, and
// read as fragments during k-block kb + 1.
//
// Work items of a k-block tile of R packed rows: R x 4 chunks of eight
// reduction indices.  With k contiguous in memory (op(A) = A, op(B) = B^T) a
// wave takes 16 rows x 4 chunks (128 contiguous bytes per row); with k strided
// a wave takes 64 consecutive rows of one chunk (256 contiguous bytes per k).
struct StreamItem {
    int row, q;
};
__device__ inline StreamItem stream_item(bool contig, int i) {
    const int t = threadIdx.x;
    return contig ? StreamItem{(t >> 2) + 64 * i, t & 3} : StreamItem{(t & 63) + 64 * i, t >> 6};
}

// Eight zeros that loads of entries outside the operand read instead.
__device__ __attribute__((aligned(16))) float g_zero8[8];

// Eight FP32 entries (packed row p, reduction indices k0 .. k0 + 7) of an
// operand stored with k contiguous (X[p ld + k]) or strided (X[k ld + p]);
// zeros outside p < plim, k < K.  An entry outside is loaded from g_zero8, so
// no condition outlives the issue of the loads (the loads of k-block kb + 3
// stay in flight across a whole k-block).  vec (k contiguous, X and ld 16-byte
// aligned, K a multiple of 8): a chunk is wholly inside or outside, read as
// two 16-byte loads.
__device__ __forceinline__ void load8_f32(const float *__restrict__ X, int64_t ld, bool contig,
                                          bool vec, int64_t p, int64_t k0, int64_t plim,
                                          int64_t K, float (&x)[8]) {
    const bool row_ok = p < plim;
    if (contig && vec) {
        const float *src = (row_ok && k0 < K) ? X + p * ld + k0 : g_zero8;
        const float4 v0 = reinterpret_cast<const float4 *>(src)[0];
        const float4 v1 = reinterpret_cast<const float4 *>(src)[1];
        x[0] = v0.x; x[1] = v0.y; x[2] = v0.z; x[3] = v0.w;
        x[4] = v1.x; x[5] = v1.y; x[6] = v1.z; x[7] = v1.w;
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float *src = (row_ok && k0 + i < K)
                                   ? X + (contig ? p * ld + k0 + i : (k0 + i) * ld + p)
                                   : g_zero8;
            x[i] = *src;
        }
    }
}

template <int RB>
__global__ __launch_bounds__(256, 1) void gemm_f32s_kernel(
    const float *__restrict__ A, int64_t lda, int a_contig, int a_vec, const float *__restrict__ B,
    int64_t ldb, int b_contig, int b_vec, float *__restrict__ C, int64_t M, int64_t N, int64_t K, int KB,
    int64_t ldc, float alpha, float beta, int nt_m, int nt_n, int kb_per_split,
    float *__restrict__ part, unsigned *__restrict__ status) {
    constexpr int MT = 64 * RB;
    constexpr int A_BYTES = MT * 64;
    constexpr int B_BYTES = NT * 64;
    constexpr int STAGE = NC * (A_BYTES + B_BYTES);
    constexpr int AI = MT / 64, BI = NT / 64;           // work items per thread and k-block
    __shared__ __attribute__((aligned(1024))) char stage0[STAGE];
    __shared__ __attribute__((aligned(1024))) char stage1[STAGE];

    int tm, tn;
    tile_coords<4>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * MT, n0 = (int64_t)tn * NT;
    const bool ca = a_contig != 0, cbn = b_contig != 0, va = a_vec != 0, vb = b_vec != 0;

    float sa[AI][8], sb[BI][8];
    unsigned st = 0;
    auto load_kb = [&](int kb) __attribute__((always_inline)) {
        const int64_t kk = (int64_t)kb * KBLK;
#pragma unroll
        for (int i = 0; i < AI; ++i) {
            const StreamItem it = stream_item(ca, i);
            load8_f32(A, lda, ca, va, m0 + it.row, kk + it.q * 8, M, K, sa[i]);
        }
#pragma unroll
        for (int i = 0; i < BI; ++i) {
            const StreamItem it = stream_item(cbn, i);
            load8_f32(B, ldb, cbn, vb, n0 + it.row, kk + it.q * 8, N, K, sb[i]);
        }
    };
    // the staged k-block's three planes of both operands into one LDS stage
    auto write_kb = [&](char *base) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AI; ++i) {
            const StreamItem it = stream_item(ca, i);
            u16x8 c0, c1, c2;
            split3_f32x8(sa[i], c0, c1, c2, st);
            char *d = base + it.row * 64 + ((it.q ^ swz(it.row)) << 4);
            *reinterpret_cast<u16x8 *>(d) = c0;
            *reinterpret_cast<u16x8 *>(d + A_BYTES) = c1;
            *reinterpret_cast<u16x8 *>(d + 2 * A_BYTES) = c2;
        }
#pragma unroll
        for (int i = 0; i < BI; ++i) {
            const StreamItem it = stream_item(cbn, i);
            u16x8 c0, c1, c2;
            split3_f32x8(sb[i], c0, c1, c2, st);
            char *d = base + NC * A_BYTES + it.row * 64 + ((it.q ^ swz(it.row)) << 4);
            *reinterpret_cast<u16x8 *>(d) = c0;
            *reinterpret_cast<u16x8 *>(d + B_BYTES) = c1;
            *reinterpret_cast<u16x8 *>(d + 2 * B_BYTES) = c2;
        }
    };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);
    struct Frags {
        bf16x8 b[NC][2];
        bf16x8 a[NC][RB];
    };
    const int at0 = (wm * 32 * RB) * 64, bt0 = NC * A_BYTES + (wn * 64) * 64;
    auto read_a = [&](const char *base, int off, int c, int rb) __attribute__((always_inline)) {
        return lds_frag(base + at0 + c * A_BYTES + rb * 32 * 64, off);
    };
    auto read_b = [&](const char *base, int off, int c, int cb) __attribute__((always_inline)) {
        return lds_frag(base + bt0 + c * B_BYTES + cb * 32 * 64, off);
    };
    // One sub-step: the product order, accumulators and fragment re-reads of
    // gemm_f32_kernel's sub-step (no copies).
    constexpr int PI[6] = {0, 0, 0, 1, 1, 2}, PJ[6] = {0, 1, 2, 0, 1, 0};
    auto step = [&](Frags &f, const bf16x8 (&b0)[2], bf16x8 (&b0n)[2], f32x16 (&hi)[RB][2],
                    f32x16 (&lo)[RB][2], auto zero_c, auto zero_lo_c, const char *nbase,
                    int noff) __attribute__((always_inline)) {
        constexpr bool zero = decltype(zero_c)::value;
        constexpr bool zero_lo = decltype(zero_lo_c)::value;
        constexpr int G = 2 * RB;
        static_for<12 * RB>([&](auto t_c) {
            constexpr int t = decltype(t_c)::value;
            constexpr int g = t / G, rb = (t % G) / 2, cb = t % 2;
            constexpr int i = PI[g], j = PJ[g];
            const bf16x8 &bop = (j == 0) ? b0[cb] : f.b[j][cb];
            if constexpr (g == 0)
                hi[rb][cb] = mfma(f.a[0][rb], bop, zero ? f32x16{} : hi[rb][cb]);
            else
                lo[rb][cb] = mfma(f.a[i][rb], bop, (zero_lo && g == 1) ? f32x16{} : lo[rb][cb]);
            order_fence();
            constexpr int ua0 = t - (2 * G + 1), ua1 = t - (4 * G + 1), ua2 = t - (5 * G + 1);
            constexpr int ub2 = t - (3 * G - 2), ub1 = t - (5 * G - 2);
            if constexpr (t < 2) b0n[t] = read_b(nbase, noff, 0, t);
            if constexpr (ua0 >= 0 && ua0 % 2 == 0 && ua0 / 2 < RB) f.a[0][ua0 / 2] = read_a(nbase, noff, 0, ua0 / 2);
            if constexpr (ub2 == 0 || ub2 == 1) f.b[2][ub2] = read_b(nbase, noff, 2, ub2);
            if constexpr (ua1 >= 0 && ua1 % 2 == 0 && ua1 / 2 < RB) f.a[1][ua1 / 2] = read_a(nbase, noff, 1, ua1 / 2);
            if constexpr (ub1 == 0 || ub1 == 1) f.b[1][ub1] = read_b(nbase, noff, 1, ub1);
            if constexpr (ua2 >= 0 && ua2 % 2 == 0 && ua2 / 2 < RB) f.a[2][ua2 / 2] = read_a(nbase, noff, 2, ua2 / 2);
            order_fence();
        });
    };

    f32x16 blk[RB][2];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) blk[i][j] = f32x16{};

    const int kb_lo = blockIdx.y * kb_per_split;
    const int kb_hi = min(KB, kb_lo + kb_per_split);
    // prologue: k-blocks kb_lo and kb_lo + 1 into the two stages, kb_lo + 2 staged
    load_kb(kb_lo);
    write_kb(stage0);
    if (kb_lo + 1 < kb_hi) {
        load_kb(kb_lo + 1);
        write_kb(stage1);
    }
    if (kb_lo + 2 < kb_hi) load_kb(kb_lo + 2);
    __syncthreads();
    Frags f;
    bf16x8 b0a[2], b0b[2];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) f.b[c][cb] = read_b(stage0, off0, c, cb);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) f.a[c][rb] = read_a(stage0, off0, c, rb);
    }
    b0a[0] = f.b[0][0];
    b0a[1] = f.b[0][1];
    int kb = kb_lo;
    f32x16 lo[RB][2];
    for (int p0 = kb_lo; p0 < kb_hi; p0 += KB_PER_PANEL) {
        const int p1 = min(kb_hi, p0 + KB_PER_PANEL);
        f32x16 hi[RB][2];
        auto kblock = [&](auto first_c, auto first_lo_c) __attribute__((always_inline)) {
            char *cur = (kb & 1) ? stage1 : stage0;
            char *nxt = (kb & 1) ? stage0 : stage1;
            step(f, b0a, b0b, hi, lo, first_c, first_lo_c, cur, off1);
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            pipeline_barrier();
            // every wave is done with stage cur: the staged k-block kb + 2 goes
            // there, and k-block kb + 3 is loaded
            if (kb + 2 < kb_hi) {
                write_kb(cur);
                if (kb + 3 < kb_hi) load_kb(kb + 3);
            }
            __builtin_amdgcn_sched_barrier(0);
            step(f, b0b, b0a, hi, lo, std::false_type{}, std::false_type{}, nxt, off0);
            __builtin_amdgcn_sched_barrier(0);
        };
        if (p0 == kb_lo) kblock(std::true_type{}, std::true_type{});
        else kblock(std::true_type{}, std::false_type{});
        for (++kb; kb < p1; ++kb) kblock(std::false_type{}, std::false_type{});
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) blk[i][j] += hi[i][j];
    }
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) blk[i][j] += lo[i][j];
    for (int off = 32; off > 0; off >>= 1) st |= __shfl_xor(st, off);
    if (lane == 0 && st) atomicOr(status, st);

#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int64_t col = n0 + wn * 64 + cb * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 32 * RB + rb * 32 + acc_row(lane, r);
                if (row < M && col < N) {
                    if (part != nullptr)
                        part[((int64_t)blockIdx.y * M + row) * N + col] = blk[rb][cb][r];
                    else
                        C[row * ldc + col] = out_update(blk[rb][cb][r], alpha, beta, C + row * ldc + col);
                }
            }
        }
}

// Split-K combination: C = alpha (sum of the splits' partial sums, in split
// order, FP32) + beta C, with the output update of the single-pass kernel.
__global__ void reduce_splits_kernel(const float *__restrict__ part, int splits, int64_t M,
                                     int64_t N, float *__restrict__ C, int64_t ldc, float alpha,
                                     float beta) {
    const int64_t total = M * N;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        float p = part[i];
        for (int sp = 1; sp < splits; ++sp) p += part[sp * total + i];
        const int64_t row = i / N, col = i - row * N;
        C[row * ldc + col] = out_update(p, alpha, beta, C + row * ldc + col);
    }
}

}  // namespace

int sgemm_splits(int64_t M, int64_t N, int64_t KB, int tile_m) {
    const int64_t cus = device_cu_count();
    const int64_t tiles = ((M + tile_m - 1) / tile_m) * ((N + NT - 1) / NT);
    const int64_t panels = (KB + KB_PER_PANEL - 1) / KB_PER_PANEL;
    // split only when the tiles fill at most half of the CUs, and keep all
    // splits within one wave of workgroups (the partial sums cost a pass)
    if (2 * tiles > cus || panels < 2) return 1;
    int64_t sp = cus / tiles;
    sp = sp < panels ? sp : panels;
    sp = sp < 16 ? sp : 16;
    const int64_t per = (panels + sp - 1) / sp;             // whole panels per split
    return (int)((panels + per - 1) / per);
}

int sgemm_tile_m(int64_t M, int64_t N, int64_t KB) {
    // One workgroup per CU runs at a time (120 or 96 KB of LDS).  Model the
    // time of each tile height as rounds of workgroups x rows per tile x
    // k-blocks per split, the 128-row tile's larger copy share per MFMA counted
    // as 5 %, and take the shorter (measured: 128 rows are 18-28 % faster at
    // 2048^3 and 2560^3, 4-13 % at 1024^3, 4096^3 and 1024 x 1024 x 65536;
    // 192 rows 2-19 % faster at 3072^3, 6144^3, 16384 x 16384 x 512 and
    // 3000 x 2000 x 4000).
    const int64_t cus = device_cu_count();
    double best = 0.0;
    int pick = 192;
    for (int t : {192, 128}) {
        const int64_t tiles = ((M + t - 1) / t) * ((N + NT - 1) / NT);
        const int64_t sp = sgemm_splits(M, N, KB, t);
        const int64_t rounds = (tiles * sp + cus - 1) / cus;
        const double cost = (double)rounds * t * (double)((KB + sp - 1) / sp) * (t == 128 ? 1.05 : 1.0);
        if (t == 192 || cost < best) {
            best = cost;
            pick = t;
        }
    }
    return pick;
}

hipError_t launch_gemm_f32(const uint16_t *Ap, const uint16_t *Bp, float *C, int64_t M, int64_t N,
                           int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, float alpha,
                           float beta, int tile_m, int splits, float *part, hipStream_t s) {
    if (tile_m != 192 && tile_m != 128) return hipErrorInvalidValue;
    const int nt_m = (int)((M + tile_m - 1) / tile_m), nt_n = (int)((N + NT - 1) / NT);
    const int64_t panels = (KB + KB_PER_PANEL - 1) / KB_PER_PANEL;
    const int kb_per_split = (int)((panels + splits - 1) / splits) * KB_PER_PANEL;
    if (splits < 1 || (splits > 1 && !part) || (int64_t)(splits - 1) * kb_per_split >= KB)
        return hipErrorInvalidValue;
    const dim3 grid(nt_m * nt_n, splits);
    float *pp = splits > 1 ? part : nullptr;
    if (tile_m == 192)
        gemm_f32_kernel<3><<<grid, 256, 0, s>>>(Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, alpha,
                                                beta, nt_m, nt_n, kb_per_split, pp);
    else
        gemm_f32_kernel<2><<<grid, 256, 0, s>>>(Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, alpha,
                                                beta, nt_m, nt_n, kb_per_split, pp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    const int64_t total = M * N;
    const int g = (int)((total + 255) / 256 < 8192 ? (total + 255) / 256 : 8192);
    reduce_splits_kernel<<<g, 256, 0, s>>>(part, splits, M, N, C, ldc, alpha, beta);
    return hipGetLastError();
}

hipError_t launch_gemm_f32_streamed(const float *A, int64_t lda, bool ta, const float *B,
                                    int64_t ldb, bool tb, float *C, int64_t M, int64_t N,
                                    int64_t K, int64_t ldc, float alpha, float beta, int splits,
                                    float *part, unsigned *status, hipStream_t s) {
    constexpr int TM = 128;
    const int64_t KB = (K + KBLK - 1) / KBLK;
    const int nt_m = (int)((M + TM - 1) / TM), nt_n = (int)((N + NT - 1) / NT);
    const int64_t panels = (KB + KB_PER_PANEL - 1) / KB_PER_PANEL;
    const int kb_per_split = (int)((panels + splits - 1) / splits) * KB_PER_PANEL;
    if (splits < 1 || (splits > 1 && !part) || (int64_t)(splits - 1) * kb_per_split >= KB)
        return hipErrorInvalidValue;
    const dim3 grid(nt_m * nt_n, splits);
    float *pp = splits > 1 ? part : nullptr;
    // k contiguous in memory: op(A) = A (row-major M x K), op(B) = B^T (B stored N x K)
    auto vec = [&](const float *X, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(X) & 15u) == 0 && ld % 4 == 0 && K % 8 == 0 ? 1 : 0;
    };
    gemm_f32s_kernel<2><<<grid, 256, 0, s>>>(A, lda, ta ? 0 : 1, vec(A, lda), B, ldb, tb ? 1 : 0,
                                             vec(B, ldb), C, M, N, K, (int)KB, ldc, alpha, beta,
                                             nt_m, nt_n, kb_per_split, pp, status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    const int64_t total = M * N;
    const int g = (int)((total + 255) / 256 < 8192 ? (total + 255) / 256 : 8192);
    reduce_splits_kernel<<<g, 256, 0, s>>>(part, splits, M, N, C, ldc, alpha, beta);
    return hipGetLastError();
}

}  // namespace emu
