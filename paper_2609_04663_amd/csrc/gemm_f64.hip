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
// straight into LDS (global_load_lds_dwordx4) through a ring of LDS stages.
// Each wave keeps one FP32 accumulator set per product for the whole panel
// (all N_p live, so every fragment read from LDS feeds every product that
// uses it) and an FP64 accumulator tile.
#include "gemm_common.h"

namespace emu {
namespace {

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER>
struct Cfg {
    static constexpr int P = D * (D + 1) / 2;       // retained products N_p(d)
    // FP64 accumulator tile in LDS instead of registers (frees 32 BM VGPRs for
    // the N_p FP32 accumulator sets; touched once per panel)
    static constexpr int ACC64_BYTES = ACC64_LDS ? 4 * 64 * 16 * BM * 8 : 0;
    // products q >= Q_VGPR keep their accumulators in VGPRs (inline-asm MFMA)
    // so that all N_p sets fit: 256 AGPRs hold 16 sets of 16 registers
    static constexpr int Q_VGPR = P * BM > 16 ? 16 / BM : P;
    static constexpr int MT = 64 * BM, NT = DGEMM_NT;
    static constexpr int A_BYTES = MT * 64, B_BYTES = NT * 64;
    static constexpr int STAGE = D * (A_BYTES + B_BYTES);
    static constexpr int NSTAGE = NS;               // LDS stages (copy lead = NS - 1 k-blocks)
    static constexpr int A_PARTS = A_BYTES / 1024, B_PARTS = B_BYTES / 1024;
    static constexpr int COPIES = D * (A_PARTS + B_PARTS) / 4;   // 1 KB copies per wave per k-block
    static constexpr int COPIES_AFTER = AFTER < COPIES ? AFTER : COPIES;
    static constexpr int READS = D * (BM + 1);      // fragment reads per sub-step
    static constexpr int MMAS = P * BM;             // MFMAs per sub-step
    static_assert(A_PARTS == 4 * BM && B_PARTS == 4, "copy split assumes 4 waves");
    static_assert(NS * STAGE + ACC64_BYTES <= 160 * 1024, "LDS");
};

// Product q = l (l + 1) / 2 + i of the retained set is A_i B_(l - i): q
// ascending is the FP64 order of Eq. (fp64reconstruction) (diagonal l
// ascending, i ascending inside a diagonal).
constexpr int diag_of(int q) {
    int l = 0;
    while ((l + 1) * (l + 2) / 2 <= q) ++l;
    return l;
}
constexpr int prod_i(int q) { return q - diag_of(q) * (diag_of(q) + 1) / 2; }
constexpr int prod_j(int q) { return diag_of(q) - prod_i(q); }

// Per sub-step instruction order.  MFMA t is product t / BM on row block
// t % BM (products in q order); read t loads the t-th distinct operand
// fragment in order of first use by that MFMA sequence, encoded as
// 64 * is_B + 8 * plane + row block.  Reads of the next sub-step go out in
// the order its MFMAs will want them.
template <int D, int BM>
constexpr int read_code(int t) {
    bool seen_a[6][4] = {}, seen_b[6] = {};
    int r = 0;
    for (int u = 0; u < D * (D + 1) / 2 * BM; ++u) {
        const int q = u / BM, b = u % BM, i = prod_i(q), j = prod_j(q);
        if (!seen_a[i][b]) {
            seen_a[i][b] = true;
            if (r++ == t) return 8 * i + b;
        }
        if (!seen_b[j]) {
            seen_b[j] = true;
            if (r++ == t) return 64 + 8 * j;
        }
    }
    return -1;
}

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER>
__global__ __launch_bounds__(256, 1) void gemm_f64_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, double *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
    const int *__restrict__ sa, const int *__restrict__ sb, double alpha, double beta, int nt_m,
    int nt_n) {
    using K = Cfg<D, BM, NS, ACC64_LDS, AFTER>;
    __shared__ __attribute__((aligned(1024))) char lds[K::NSTAGE * K::STAGE + K::ACC64_BYTES];
    // lane-private FP64 accumulators in LDS: element r of lane l of wave w at
    // ((w * BM + b) * 16 + r) * 64 + l (consecutive lanes, consecutive doubles)
    double *acc64_lds = reinterpret_cast<double *>(lds + K::NSTAGE * K::STAGE);

    int tm, tn;
    tile_coords<8>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const unsigned lane16 = (unsigned)lane * 16u;   // copy offset of this lane
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * K::MT, n0 = (int64_t)tn * K::NT;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = (int64_t)KB * RpadA * 64;
    const int64_t b_plane = (int64_t)KB * RpadB * 64;

    // Copy issue for one k-block: wave w moves 1 KB parts [w BM, (w + 1) BM) of
    // every A plane and part w of every B plane (wave-uniform base plus
    // compile-time offsets).
    const int64_t a_base = m0 * 64 + (int64_t)wave * BM * 1024;
    const int64_t b_base = n0 * 64 + (int64_t)wave * 1024;
    // Copy j of a k-block (j < COPIES) moves plane c = j / (BM + 1), A part
    // j % (BM + 1) (or the B part when that is BM).
    auto issue_one = [&](int kb, char *base, auto j_c) {
        constexpr int j = decltype(j_c)::value, c = j / (BM + 1), r = j % (BM + 1);
        if constexpr (r < BM)
            copy_1k(Ag + (int64_t)kb * RpadA * 64 + a_base + c * a_plane + r * 1024,
                    base + wave * BM * 1024 + c * K::A_BYTES + r * 1024, lane16);
        else
            copy_1k(Bg + (int64_t)kb * RpadB * 64 + b_base + c * b_plane,
                    base + D * K::A_BYTES + wave * 1024 + c * K::B_BYTES, lane16);
    };
    auto issue_all = [&](int kb, char *base) {
        static_for<K::COPIES>([&](auto j_c) { issue_one(kb, base, j_c); });
    };
    // copies issued after the mid-k-block barrier; the rest go out before it
    constexpr int H0 = K::COPIES_AFTER;
    auto stage = [&](int kb) -> char * { return lds + (kb % K::NSTAGE) * K::STAGE; };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);

    // Fragments of one 16-index sub-step: D planes of A (BM row blocks) and of B.
    struct Frags {
        bf16x8 a[D][BM], b[D];
    };
    const char *const At0 = lds + (wm * 32 * BM) * 64;
    const char *const Bt0 = lds + D * K::A_BYTES + (wn * 32) * 64;
    auto load = [&](int stage_off, int off, Frags &f) {
#pragma unroll
        for (int m = 0; m < D; ++m) {
            f.b[m] = lds_frag(Bt0 + stage_off + m * K::B_BYTES, off);
#pragma unroll
            for (int b = 0; b < BM; ++b)
                f.a[m][b] = lds_frag(At0 + stage_off + m * K::A_BYTES + b * 32 * 64, off);
        }
    };
    // One sub-step: the MMAS MFMAs on `cur`, the READS fragment reads of the
    // next sub-step (stage offset nso, lane offset noff) into `nxt`, and copies
    // [J0, J1) of k-block ckb into stage cdst, in slots of one MFMA, one read and
    // one copy (MFMA first: its operands were read a sub-step earlier), so that
    // reads and copies are issued while MFMAs execute.  The accumulator order
    // (q) encodes the FP64 addition order; the MFMA order inside a panel does
    // not matter (exact panel sums).
    constexpr int SLOTS = K::MMAS > K::READS ? K::MMAS : K::READS;
    auto step = [&](const Frags &cur, f32x16 (&acc)[K::P][BM], auto zero_c, int nso, int noff,
                    Frags &nxt, int ckb, char *cdst, auto j0_c, auto j1_c) {
        constexpr bool zero = decltype(zero_c)::value;
        constexpr int J0 = decltype(j0_c)::value, J1 = decltype(j1_c)::value;
        static_for<(SLOTS > J1 - J0 ? SLOTS : J1 - J0)>([&](auto t_c) {
            constexpr int t = decltype(t_c)::value;
            if constexpr (t < K::MMAS) {
                constexpr int q = t / BM, b = t % BM, i = prod_i(q), j = prod_j(q);
                if constexpr (q >= K::Q_VGPR) {
                    if constexpr (zero) mfma_vacc_zero(acc[q][b], cur.a[i][b], cur.b[j]);
                    else mfma_vacc(acc[q][b], cur.a[i][b], cur.b[j]);
                } else {
                    acc[q][b] = mfma(cur.a[i][b], cur.b[j], zero ? f32x16{} : acc[q][b]);
                }
            }
            order_fence();
            if constexpr (t < K::READS) {
                constexpr int code = read_code<D, BM>(t);
                constexpr int plane = (code >> 3) & 7, blk = code & 7;
                if constexpr (code >= 64)
                    nxt.b[plane] = lds_frag(Bt0 + nso + plane * K::B_BYTES, noff);
                else
                    nxt.a[plane][blk] = lds_frag(At0 + nso + plane * K::A_BYTES + blk * 32 * 64, noff);
            }
            order_fence();
            if constexpr (t < J1 - J0) issue_one(ckb, cdst, std::integral_constant<int, J0 + t>{});
            order_fence();
        });
    };

    double acc64[ACC64_LDS ? 1 : BM][16];
#pragma unroll
    for (int b = 0; b < BM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if constexpr (ACC64_LDS)
                acc64_lds[((wave * BM + b) * 16 + r) * 64 + lane] = 0.0;
            else
                acc64[b][r] = 0.0;
        }

    // Software pipeline over k-blocks with a ring of NS LDS stages (stage of
    // k-block kb: kb mod NS).  The copy of k-block kb + NS goes to stage kb,
    // which is free once trip kb's mid barrier has passed: its first H0 copies
    // are issued right after that barrier, the rest in trip kb + 1 before its
    // barrier.  Trip kb (1) reads the sub-step-1 fragments of kb while the
    // sub-step-0 MFMAs run, and issues the remaining copies of k-block
    // kb + NS - 1; (2) waits until at most the newest NS - 2 k-blocks of its own
    // copies are outstanding (so kb + 1 has landed) and for its LDS reads, then
    // barriers: every wave is done reading stage kb and every copy of kb + 1 has
    // landed; (3) issues the first H0 copies of k-block kb + NS into stage kb and
    // reads the sub-step-0 fragments of kb + 1 while the sub-step-1 MFMAs run.
    // Copies past the last k-block re-read the last one (in bounds, never used).
    for (int j = 0; j < K::NSTAGE - 1; ++j) issue_all(min(j, KB - 1), stage(j));
    static_for<H0>([&](auto j_c) { issue_one(min(K::NSTAGE - 1, KB - 1), stage(K::NSTAGE - 1), j_c); });
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((K::NSTAGE - 2) * K::COPIES + H0) : "memory");
    __syncthreads();
    Frags f0, f1;
    load(0, off0, f0);
    int kb = 0;
    for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
        const int p1 = min(KB, p0 + KB_PER_PANEL);
        f32x16 acc[K::P][BM];
        auto kblock = [&](auto first_c) {
            const int so = (kb % K::NSTAGE) * K::STAGE;
            const int nso = ((kb + 1) % K::NSTAGE) * K::STAGE;
            // sub-step 0 of kb; reads sub-step 1 of kb
            step(f0, acc, first_c, so, off1, f1, min(kb + K::NSTAGE - 1, KB - 1),
                 stage(kb + K::NSTAGE - 1), std::integral_constant<int, H0>{},
                 std::integral_constant<int, K::COPIES>{});
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (K::NSTAGE == 2)
                asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            else
                asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"((K::NSTAGE - 2) * K::COPIES)
                             : "memory");
            pipeline_barrier();
            // sub-step 1 of kb; reads sub-step 0 of kb + 1
            step(f1, acc, std::false_type{}, nso, off0, f0, min(kb + K::NSTAGE, KB - 1), lds + so,
                 std::integral_constant<int, 0>{}, std::integral_constant<int, H0>{});
            __builtin_amdgcn_sched_barrier(0);
        };
        kblock(std::true_type{});
        for (++kb; kb < p1; ++kb) kblock(std::false_type{});
        // panel end: widen each product exactly and add it in FP64, in order
#pragma unroll
        for (int q = K::Q_VGPR; q < K::P; ++q)
#pragma unroll
            for (int b = 0; b < BM; ++b) mfma_vacc_settle(acc[q][b]);
        if constexpr (ACC64_LDS) {
            // eight elements at a time: eight independent FP64 chains keep the
            // FP64 adder busy (one element's 21 adds in a row would wait on
            // each other)
#pragma unroll
            for (int b = 0; b < BM; ++b)
#pragma unroll
                for (int h = 0; h < 16; h += 8) {
                    double t[8];
#pragma unroll
                    for (int r = 0; r < 8; ++r)
                        t[r] = acc64_lds[((wave * BM + b) * 16 + h + r) * 64 + lane];
#pragma unroll
                    for (int q = 0; q < K::P; ++q)
#pragma unroll
                        for (int r = 0; r < 8; ++r) t[r] += (double)acc[q][b][h + r];
#pragma unroll
                    for (int r = 0; r < 8; ++r)
                        acc64_lds[((wave * BM + b) * 16 + h + r) * 64 + lane] = t[r];
                }
        } else {
#pragma unroll
            for (int q = 0; q < K::P; ++q)
#pragma unroll
                for (int b = 0; b < BM; ++b)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc64[b][r] += (double)acc[q][b][r];
        }
    }
    // the last trips issued (unused) copies: let them land before the workgroup
    // ends and its LDS is handed to another workgroup
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // store; with the scale-aware split the row and column weights go back in
    // here, C_mn = 2^(sa_m + sb_n) C'_mn (exact up to overflow or underflow)
    const int col_w = (sa != nullptr && n0 + wn * 32 + (lane & 31) < N) ? sb[n0 + wn * 32 + (lane & 31)] : 0;
#pragma unroll
    for (int b = 0; b < BM; ++b) {
        const int64_t col = n0 + wn * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = m0 + wm * 32 * BM + b * 32 + acc_row(lane, r);
            if (row < M && col < N) {
                double val = ACC64_LDS ? acc64_lds[((wave * BM + b) * 16 + r) * 64 + lane]
                                       : acc64[ACC64_LDS ? 0 : b][r];
                if (sa != nullptr) val = ldexp(val, sa[row] + col_w);
                C[row * ldc + col] = out_update(val, alpha, beta, C + row * ldc + col);
            }
        }
    }
}

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER>
hipError_t launch_t(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M, int64_t N,
                    int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, const int *sa,
                    const int *sb, double alpha, double beta, hipStream_t s) {
    using K = Cfg<D, BM, NS, ACC64_LDS, AFTER>;
    const int nt_m = (int)((M + K::MT - 1) / K::MT), nt_n = (int)((N + K::NT - 1) / K::NT);
    gemm_f64_kernel<D, BM, NS, ACC64_LDS, AFTER><<<nt_m * nt_n, 256, 0, s>>>(Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc,
                                                       sa, sb, alpha, beta, nt_m, nt_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_f64(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M,
                           int64_t N, int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
                           const int *sa, const int *sb, double alpha, double beta, int d,
                           hipStream_t s) {
    switch (d) {
        case 3: return launch_t<3, 2, 3, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 4: return launch_t<4, 1, 3, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 5: return launch_t<5, 1, 3, true, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 6: return launch_t<6, 1, 2, true, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace emu
