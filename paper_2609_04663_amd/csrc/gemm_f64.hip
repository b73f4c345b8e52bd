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
// Two kernels.  gemm_f64_kernel (below): 32 x 32 x 16 MFMA, 4 waves in a 2 x 2
// grid; wave tile (32 BM) x 32, output tile (64 BM) x 64.  gemm_f64w_kernel
// (further down): 16 x 16 x 32 MFMA on a (16 BMW) x 32 wave tile, one barrier
// per k-block; it runs depths d >= 6 (BMW = 1) and, with BMW = 2 or 4, the
// long reductions of d = 1, 2, 4, 5 and the small grids of d = 1 .. 3 (the
// choice is made in launch_gemm_f64).  Per k-block of 32 the d planes of both operands are copied
// straight into LDS (global_load_lds_dwordx4) through a ring of LDS stages.
// Each wave keeps one FP32 accumulator set per product for the whole panel
// (all N_p live, so every fragment read from LDS feeds every product that
// uses it) and an FP64 accumulator tile.
#include "gemm_common.h"

namespace emu {
namespace {

// Product q of the retained set S_d of Eq. (product-selection), in executed
// order: diagonal l = i + j ascending, i ascending inside a diagonal, slice
// indices i, j < 6.  q ascending is the FP64 order of Eq. (fp64reconstruction);
// the sets of the depths d are prefixes of one sequence (for d <= 6 product q
// is A_i B_(l - i) with q = l (l + 1) / 2 + i).
constexpr int pair_code(int q) {
    int n = 0;
    for (int l = 0; l < 11; ++l)
        for (int i = (l > 5 ? l - 5 : 0); i <= (l < 5 ? l : 5); ++i)
            if (n++ == q) return 8 * i + (l - i);
    return -1;
}
constexpr int prod_i(int q) { return pair_code(q) >> 3; }
constexpr int prod_j(int q) { return pair_code(q) & 7; }
constexpr int n_prod(int d) {
    int n = 0;
    for (int i = 0; i < 6; ++i)
        for (int j = 0; j < 6; ++j) n += (i + j < d);
    return n;
}

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER>
struct Cfg {
    static constexpr int P = n_prod(D);             // retained products N_p(d)
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

// Per sub-step instruction order.  MFMA t is product t / BM on row block
// t % BM (products in q order); read t loads the t-th distinct operand
// fragment in order of first use by that MFMA sequence, encoded as
// 64 * is_B + 8 * plane + row block.  Reads of the next sub-step go out in
// the order its MFMAs will want them.
template <int D, int BM>
constexpr int read_code(int t) {
    bool seen_a[6][4] = {}, seen_b[6] = {};
    int r = 0;
    for (int u = 0; u < n_prod(D) * BM; ++u) {
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

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER, bool PERSIST>
__global__ __launch_bounds__(256, 1) void gemm_f64_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, double *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
    const int *__restrict__ sa, const int *__restrict__ sb, double alpha, double beta, int nt_m,
    int nt_n, int ntiles) {
    using K = Cfg<D, BM, NS, ACC64_LDS, AFTER>;
    static_assert(K::COPIES_AFTER == K::COPIES, "one k-block's copies per trip (cursor below)");
    __shared__ __attribute__((aligned(1024))) char lds[K::NSTAGE * K::STAGE + K::ACC64_BYTES];
    // lane-private FP64 accumulators in LDS: element r of lane l of wave w at
    // ((w * BM + b) * 16 + r) * 64 + l (consecutive lanes, consecutive doubles)
    double *acc64_lds = reinterpret_cast<double *>(lds + K::NSTAGE * K::STAGE);

    // PERSIST: workgroup w0 of G takes tiles w0, w0 + G, ... (`mine` of them)
    // and walks them as one sequence of k-blocks, the copies running on into
    // the next tile; otherwise one tile per workgroup.
    const int G = gridDim.x;
    const int mine = PERSIST ? (ntiles - 1 - (int)blockIdx.x) / G + 1 : 1;
    const int lane = threadIdx.x & 63;
    const unsigned lane16 = (unsigned)lane * 16u;   // copy offset of this lane
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int wm = wave >> 1, wn = wave & 1;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = plane_elems(KB, RpadA) * 2;
    const int64_t b_plane = plane_elems(KB, RpadB) * 2;

    // Copy issue for one k-block: wave w moves 1 KB parts [w BM, (w + 1) BM) of
    // every A plane and part w of every B plane (wave-uniform base plus
    // compile-time offsets).  ak, bk: the k-block's slab of plane 0 at the
    // copied tile's first row.
    const int64_t a_base = (int64_t)wave * BM * 1024;
    const int64_t b_base = (int64_t)wave * 1024;
    // Copy j of a k-block (j < COPIES) moves plane c = j / (BM + 1), A part
    // j % (BM + 1) (or the B part when that is BM).
    auto issue_one = [&](const char *ak, const char *bk, char *base, auto j_c) {
        constexpr int j = decltype(j_c)::value, c = j / (BM + 1), r = j % (BM + 1);
        if constexpr (r < BM)
            copy_1k(ak + a_base + c * a_plane + r * 1024,
                    base + wave * BM * 1024 + c * K::A_BYTES + r * 1024, lane16);
        else
            copy_1k(bk + b_base + c * b_plane, base + D * K::A_BYTES + wave * 1024 + c * K::B_BYTES,
                    lane16);
    };
    // Copy cursor: the (tile, k-block) the next copies fetch; past the last
    // k-block of the last tile it stays on that k-block (in bounds, unused).
    int c_tile = 0, c_kb = 0;
    const char *c_ak, *c_bk;
    // tiles in groups of 4 tile-rows per XCD (the tiles of this kernel are up
    // to four times taller than wide; measured 1-10 % less time than groups
    // of 8 at 16384 x 16384 x 512 and 8192 x 8192 x 1024)
    auto cursor_bases = [&]() {
        int tm, tn;
        tile_coords_of<4>((int)blockIdx.x + c_tile * G, ntiles, nt_m, nt_n, tm, tn);
        c_ak = Ag + (int64_t)c_kb * RpadA * 64 + (int64_t)tm * K::MT * 64;
        c_bk = Bg + (int64_t)c_kb * RpadB * 64 + (int64_t)tn * K::NT * 64;
    };
    auto cursor_next = [&]() {
        if (c_kb + 1 < KB) {
            ++c_kb;
            c_ak += RpadA * 64;
            c_bk += RpadB * 64;
        } else if (PERSIST && c_tile + 1 < mine) {
            ++c_tile;
            c_kb = 0;
            cursor_bases();
        }
    };
    auto stage = [&](int qs) -> char * { return lds + qs * K::STAGE; };

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
                    Frags &nxt, const char *ak, const char *bk, char *cdst, auto j0_c, auto j1_c) {
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
            if constexpr (t < J1 - J0)
                issue_one(ak, bk, cdst, std::integral_constant<int, J0 + t>{});
            order_fence();
        });
    };

    // Software pipeline over the workgroup's sequence of k-blocks with a ring of
    // NS LDS stages (position q in stage q mod NS).  Trip q (1) reads the
    // sub-step-1 fragments of q while the sub-step-0 MFMAs run; (2) waits until
    // at most the newest NS - 2 k-blocks of its own copies are outstanding (so
    // q + 1 has landed) and for its LDS reads, then barriers: every wave is done
    // reading stage q and every copy of q + 1 has landed; (3) issues the copies
    // of q + NS into stage q and reads the sub-step-0 fragments of q + 1 while
    // the sub-step-1 MFMAs run.  Across a tile boundary q + 1 is the next tile's
    // first k-block, already in place.
    cursor_bases();
    for (int j = 0; j < K::NSTAGE; ++j) {
        static_for<K::COPIES>([&](auto j_c) { issue_one(c_ak, c_bk, stage(j), j_c); });
        cursor_next();
    }
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((K::NSTAGE - 2) * K::COPIES + K::COPIES) : "memory");
    __syncthreads();
    Frags f0, f1;
    load(0, off0, f0);
    int qs = 0;                        // q mod NS
    auto kblock = [&](f32x16 (&acc)[K::P][BM], auto first_c) {
        const int so = qs * K::STAGE;
        const int qn = qs + 1 == K::NSTAGE ? 0 : qs + 1;
        // sub-step 0 of q; reads sub-step 1 of q
        step(f0, acc, first_c, so, off1, f1, c_ak, c_bk, stage(qs),
             std::integral_constant<int, K::COPIES>{}, std::integral_constant<int, K::COPIES>{});
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (K::NSTAGE == 2)
            asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
        else
            asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"((K::NSTAGE - 2) * K::COPIES)
                         : "memory");
        pipeline_barrier();
        // sub-step 1 of q; reads sub-step 0 of q + 1; copies of q + NS into stage q
        step(f1, acc, std::false_type{}, qn * K::STAGE, off0, f0, c_ak, c_bk, stage(qs),
             std::integral_constant<int, 0>{}, std::integral_constant<int, K::COPIES>{});
        __builtin_amdgcn_sched_barrier(0);
        cursor_next();
        qs = qn;
    };

    for (int it = 0; it < mine; ++it) {
        int tm, tn;
        tile_coords_of<4>((int)blockIdx.x + it * G, ntiles, nt_m, nt_n, tm, tn);
        const int64_t m0 = (int64_t)tm * K::MT, n0 = (int64_t)tn * K::NT;
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
        for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
            const int p1 = min(KB, p0 + KB_PER_PANEL);
            f32x16 acc[K::P][BM];
            kblock(acc, std::true_type{});
            for (int kb = p0 + 1; kb < p1; ++kb) kblock(acc, std::false_type{});
            // panel end: widen each product exactly and add it in FP64, in order
#pragma unroll
            for (int q = K::Q_VGPR; q < K::P; ++q)
#pragma unroll
                for (int b = 0; b < BM; ++b) mfma_vacc_settle(acc[q][b]);
            if constexpr (ACC64_LDS) {
                // eight elements at a time: eight independent FP64 chains keep
                // the FP64 adder busy (one element's 21 adds in a row would wait
                // on each other)
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

        // store; with the scale-aware split the row and column weights go back
        // in here, C_mn = 2^(sa_m + sb_n) C'_mn (exact up to overflow or underflow)
        const int col_w =
            (sa != nullptr && n0 + wn * 32 + (lane & 31) < N) ? sb[n0 + wn * 32 + (lane & 31)] : 0;
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
    // the last trips issued (unused) copies: let them land before the workgroup
    // ends and its LDS is handed to another workgroup
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------------------
// Depths d = 6 .. 11 (21 .. 36 products, every slice of both operands).  For
// d >= 7 a 32 x 32 wave tile would need 16 N_p accumulator registers per lane,
// more than the register file holds, so these depths use the 16 x 16 x 32 MFMA
// on a 16 x 32 wave tile (BMW = 1: two 16 x 16 blocks along N): 8 registers
// per product.  Workgroup: 4 waves in a 2 x 2 grid, output tile 32 x 64; one
// k-block of 32 reduction indices (one MFMA depth) per trip and one barrier
// per trip, with the copies and fragment reads spread over the trip's MFMAs
// and copies issued two trips ahead.  d = 6 runs here too: measured at
// M = N = K = 8192 it is about 5 % faster than on the 32 x 32 kernel.
// Depths d <= 5 (d planes per operand) can take a 32 x 32 wave tile here
// (BMW = 2: 2 x 2 blocks, 16 registers per product, output tile 64 x 64) or,
// with few products, 64 x 32 (BMW = 4, output tile 128 x 64).
template <int D, int NS, bool ACC64_LDS, int BMW>
struct CfgW {
    static constexpr int P = n_prod(D);
    static constexpr int NPL = D < 6 ? D : 6;                        // slices read per operand
    // FP64 accumulator tile in LDS (8 BMW doubles per lane) instead of VGPRs
    static constexpr int ACC64_BYTES = ACC64_LDS ? 4 * 64 * 8 * BMW * 8 : 0;
    static constexpr int MT = 32 * BMW, NT = 64;                     // wave tile 16 BMW x 32
    static constexpr int A_BYTES = MT * 64, B_BYTES = NT * 64;       // one plane of a stage
    static constexpr int STAGE = NPL * (A_BYTES + B_BYTES);
    static constexpr int COPIES = STAGE / 1024 / 4;                  // 1 KB copies per wave
    static constexpr int A_COPIES = NPL * MT / 16 / 4;               // the first ones move A
    static constexpr int READS = NPL * (BMW + 2);                    // A: BMW blocks, B: 2
    static constexpr int MMAS = 2 * BMW * P;
    // AGPRs hold 32 / BMW products of 2 BMW blocks; later products use VGPRs
    static constexpr int Q_VGPR = P > 32 / BMW ? 32 / BMW : P;
    static_assert(BMW == 1 || BMW == 2 || BMW == 4, "wave tile");
    static_assert(4 * COPIES * 1024 == STAGE && 4 * A_COPIES * 1024 == NPL * A_BYTES,
                  "copy split");
    static_assert(BMW != 1 || NPL == 6, "one-block tiles copy six planes");
    static_assert(NS * STAGE + ACC64_BYTES <= 160 * 1024, "LDS");
};

// Read t of a trip loads the t-th distinct fragment in order of first use by
// the trip's MFMA sequence (product q on block b for MFMA 2 q + b), encoded as
// 64 * is_B + 8 * plane + block.
template <int D, int BMW>
constexpr int read_code_w(int t) {
    bool seen_a[6][4] = {}, seen_b[6][2] = {};
    int r = 0;
    for (int u = 0; u < 2 * BMW * n_prod(D); ++u) {
        const int q = u / (2 * BMW), a = (u % (2 * BMW)) / 2, b = u % 2, i = prod_i(q),
                  j = prod_j(q);
        if (!seen_a[i][a]) {
            seen_a[i][a] = true;
            if (r++ == t) return 8 * i + a;
        }
        if (!seen_b[j][b]) {
            seen_b[j][b] = true;
            if (r++ == t) return 64 + 8 * j + b;
        }
    }
    return -1;
}

template <int D, int NS, bool ACC64_LDS, bool PERSIST, int BMW>
__global__ __launch_bounds__(256, 1) void gemm_f64w_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, double *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
    const int *__restrict__ sa, const int *__restrict__ sb, double alpha, double beta, int nt_m,
    int nt_n, int ntiles) {
    using K = CfgW<D, NS, ACC64_LDS, BMW>;
    __shared__ __attribute__((aligned(1024))) char lds[NS * K::STAGE + K::ACC64_BYTES];
    // lane-private FP64 accumulators in LDS: element e = 4 (2 a + b) + r of
    // lane l of wave w at (w * 8 BMW + e) * 64 + l
    double *acc64_lds = reinterpret_cast<double *>(lds + NS * K::STAGE);

    // Persistent workgroups: workgroup w0 of G takes tiles w0, w0 + G, ... (its
    // `mine` tiles), walking one sequence of k-blocks tile after tile, so the
    // copy ring runs on into the next tile's first k-blocks while a tile's
    // FP64 epilogue and store execute.
    const int G = gridDim.x;
    const int mine = PERSIST ? (ntiles - 1 - (int)blockIdx.x) / G + 1 : 1;
    const int lane = threadIdx.x & 63;
    const unsigned lane16 = (unsigned)lane * 16u;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;

    const char *Ag = reinterpret_cast<const char *>(Ap);
    const char *Bg = reinterpret_cast<const char *>(Bp);
    const int64_t a_plane = plane_elems(KB, RpadA) * 2;
    const int64_t b_plane = plane_elems(KB, RpadB) * 2;

    // Copy c of a k-block by wave w moves 1 KB part g = 4 c + w of the list
    // A parts (plane-major, 2 BMW parts a plane), then B parts: for BMW = 1,
    // c < 3 moves part (w & 1) of A plane 2 c + (w >> 1); for BMW >= 2,
    // c < A_COPIES moves part 4 (c % (BMW / 2)) + w of A plane c / (BMW / 2);
    // the rest move part w of B plane c - A_COPIES.
    // ak, bk: the k-block's slab of plane 0 at the copied tile's first row.
    const int64_t a_off = BMW == 1 ? (int64_t)(wave >> 1) * a_plane + (wave & 1) * 1024
                                   : (int64_t)wave * 1024;
    const int a_dst = BMW == 1 ? (wave >> 1) * K::A_BYTES + (wave & 1) * 1024 : wave * 1024;
    const int64_t b_off = (int64_t)wave * 1024;
    const int b_dst = K::NPL * K::A_BYTES + wave * 1024;
    auto issue_one = [&](const char *ak, const char *bk, char *base, auto c_c) {
        constexpr int c = decltype(c_c)::value;
        // compile-time part of copy c's A offsets
        constexpr int a_pl = BMW == 1 ? 2 * c : c / (BMW > 1 ? BMW / 2 : 1);
        constexpr int a_pt = BMW == 1 ? 0 : 4 * (c % (BMW > 1 ? BMW / 2 : 1));
        if constexpr (c < K::A_COPIES)
            copy_1k(ak + a_off + a_pl * a_plane + a_pt * 1024,
                    base + a_dst + a_pl * K::A_BYTES + a_pt * 1024, lane16);
        else
            copy_1k(bk + b_off + (c - K::A_COPIES) * b_plane,
                    base + b_dst + (c - K::A_COPIES) * K::B_BYTES, lane16);
    };
    // Copy cursor: the (tile, k-block) the next copies fetch; past the last
    // k-block of the last tile it stays on that k-block (in bounds, unused).
    int c_tile = 0, c_kb = 0;
    const char *c_ak, *c_bk;
    auto cursor_bases = [&]() {
        int tm, tn;
        tile_coords_of<8>((int)blockIdx.x + c_tile * G, ntiles, nt_m, nt_n, tm, tn);
        c_ak = Ag + (int64_t)c_kb * RpadA * 64 + (int64_t)tm * K::MT * 64;
        c_bk = Bg + (int64_t)c_kb * RpadB * 64 + (int64_t)tn * K::NT * 64;
    };
    auto cursor_next = [&]() {
        if (c_kb + 1 < KB) {
            ++c_kb;
            c_ak += RpadA * 64;
            c_bk += RpadB * 64;
        } else if (PERSIST && c_tile + 1 < mine) {
            ++c_tile;
            c_kb = 0;
            cursor_bases();
        }
    };
    auto stage = [&](int qs) -> char * { return lds + qs * K::STAGE; };

    // lane's fragment offset inside a 16-row block: row l % 16, chunk l / 16
    const int frow = lane & 15;
    const int foff = frow * 64 + (((lane >> 4) ^ swz(frow)) << 4);
    const char *const At0 = lds + (wm * 16 * BMW) * 64 + foff;
    const char *const Bt0 = lds + K::NPL * K::A_BYTES + (wn * 32) * 64 + foff;

    struct Frags {
        bf16x8 a[K::NPL][BMW], b[K::NPL][2];
    };
    auto read_one = [&](int so, Frags &f, auto t_c) {
        constexpr int code = read_code_w<D, BMW>(decltype(t_c)::value);
        constexpr int plane = (code >> 3) & 7, blk = code & 7;
        if constexpr (code >= 64)
            f.b[plane][blk] =
                *reinterpret_cast<const bf16x8 *>(Bt0 + so + plane * K::B_BYTES + blk * 16 * 64);
        else
            f.a[plane][blk] =
                *reinterpret_cast<const bf16x8 *>(At0 + so + plane * K::A_BYTES + blk * 16 * 64);
    };

    // One trip: the MMAS MFMAs on `cur`; read t of the next k-block (stage
    // offset nso) at slot RS t; copy c of k-block ckb into stage cdst at slot
    // CS c + 2 (reads and copies spread over the MFMA stream).
    constexpr int SLOTS = K::MMAS;
    constexpr int RS = SLOTS >= 2 * K::READS ? 2 : 1;
    constexpr int CS = (SLOTS - 2) / K::COPIES;
    static_assert(RS * (K::READS - 1) < SLOTS && CS >= 1, "slots");
    auto trip = [&](const Frags &cur, f32x4 (&acc)[K::P][2 * BMW], auto zero_c, int nso,
                    Frags &nxt, const char *ak, const char *bk, char *cdst) {
        constexpr bool zero = decltype(zero_c)::value;
        static_for<SLOTS>([&](auto t_c) {
            constexpr int t = decltype(t_c)::value;
            // product q on block e = 2 a + b (A block a, B block b)
            constexpr int q = t / (2 * BMW), e = t % (2 * BMW), a = e / 2, b = e % 2;
            constexpr int i = prod_i(q), j = prod_j(q);
            if constexpr (q >= K::Q_VGPR) {
                if constexpr (zero) mfma16_vacc_zero(acc[q][e], cur.a[i][a], cur.b[j][b]);
                else mfma16_vacc(acc[q][e], cur.a[i][a], cur.b[j][b]);
            } else {
                acc[q][e] = mfma16(cur.a[i][a], cur.b[j][b], zero ? f32x4{} : acc[q][e]);
            }
            order_fence();
            if constexpr (t % RS == 0 && t / RS < K::READS)
                read_one(nso, nxt, std::integral_constant<int, t / RS>{});
            order_fence();
            if constexpr (t >= 2 && (t - 2) % CS == 0 && (t - 2) / CS < K::COPIES)
                issue_one(ak, bk, cdst, std::integral_constant<int, (t - 2) / CS>{});
            order_fence();
        });
    };

    // Ring of NS stages; the k-block at position q of the workgroup's sequence
    // sits in stage q mod NS.  Trip q starts once every wave's copies of q + 1
    // have landed and every wave has read q into registers (one barrier); it
    // then runs the MFMAs of q, reads q + 1 and issues the copies of q + NS into
    // the stage of q.  Across a tile boundary q + 1 is the next tile's first
    // k-block, already in place, so only the first tile waits for a fill.
    cursor_bases();
    for (int j = 0; j < NS; ++j) {
        static_for<K::COPIES>([&](auto c_c) { issue_one(c_ak, c_bk, stage(j), c_c); });
        cursor_next();
    }
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 1) * K::COPIES) : "memory");
    __syncthreads();
    Frags f0, f1;
    static_for<K::READS>([&](auto t_c) { read_one(0, f0, t_c); });
    int qs = 0;                        // q mod NS
    auto one = [&](const Frags &cur, Frags &nxt, f32x4 (&acc)[K::P][2 * BMW], auto zero_c) {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"((NS - 2) * K::COPIES) : "memory");
        pipeline_barrier();
        const int qn = qs + 1 == NS ? 0 : qs + 1;
        trip(cur, acc, zero_c, qn * K::STAGE, nxt, c_ak, c_bk, stage(qs));
        __builtin_amdgcn_sched_barrier(0);
        cursor_next();
        qs = qn;
    };

    for (int it = 0; it < mine; ++it) {
        int tm, tn;
        tile_coords_of<8>((int)blockIdx.x + it * G, ntiles, nt_m, nt_n, tm, tn);
        const int64_t m0 = (int64_t)tm * K::MT, n0 = (int64_t)tn * K::NT;
        double acc64[2 * BMW][4];
#pragma unroll
        for (int e = 0; e < 2 * BMW; ++e)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                acc64[e][r] = 0.0;
                if constexpr (ACC64_LDS)
                    acc64_lds[(wave * 8 * BMW + 4 * e + r) * 64 + lane] = 0.0;
            }
        // trips alternate the fragment buffers: a panel starts on f0 (panels
        // have even length, except the last panel of a tile when KB is odd,
        // and then the workgroup has one tile)
        for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
            const int p1 = min(KB, p0 + KB_PER_PANEL);
            f32x4 acc[K::P][2 * BMW];
            int kb = p0;
            one(f0, f1, acc, std::true_type{});
            for (++kb; kb < p1; ++kb) {
                one(f1, f0, acc, std::false_type{});
                if (++kb < p1) one(f0, f1, acc, std::false_type{});
            }
            // panel end: widen each product exactly and add it in FP64, in order
#pragma unroll
            for (int q = K::Q_VGPR; q < K::P; ++q)
#pragma unroll
                for (int e = 0; e < 2 * BMW; ++e) mfma16_vacc_settle(acc[q][e]);
            // 8 BMW independent FP64 chains, products in order
            if constexpr (ACC64_LDS) {
#pragma unroll
                for (int x = 0; x < 8 * BMW; ++x)
                    acc64[x / 4][x % 4] = acc64_lds[(wave * 8 * BMW + x) * 64 + lane];
            }
#pragma unroll
            for (int q = 0; q < K::P; ++q)
#pragma unroll
                for (int e = 0; e < 2 * BMW; ++e)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc64[e][r] += (double)acc[q][e][r];
            if constexpr (ACC64_LDS) {
#pragma unroll
                for (int x = 0; x < 8 * BMW; ++x)
                    acc64_lds[(wave * 8 * BMW + x) * 64 + lane] = acc64[x / 4][x % 4];
            }
        }

#pragma unroll
        for (int e = 0; e < 2 * BMW; ++e) {
            const int a = e / 2, b = e % 2;
            const int64_t row0 = m0 + wm * 16 * BMW + a * 16 + (lane >> 4) * 4;
            const int64_t col = n0 + wn * 32 + b * 16 + (lane & 15);
            const int col_w = (sa != nullptr && col < N) ? sb[col] : 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t row = row0 + r;
                if (row < M && col < N) {
                    double val = acc64[e][r];
                    if (sa != nullptr) val = ldexp(val, sa[row] + col_w);
                    C[row * ldc + col] = out_update(val, alpha, beta, C + row * ldc + col);
                }
            }
        }
    }
    // the last trips issued (unused) copies: let them land before the workgroup
    // ends and its LDS is handed to another workgroup
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------------------
// Long reductions of depths d = 3 .. 6 on the 32 x 32 x 16 MFMA with wave tiles
// of BM 32 x 32 blocks: four waves in a 2 x 2 grid, output tile (64 BM) x 64
// (d = 6 and 5: BM = 1; d = 4 and 3: BM = 2).  Every retained product's
// accumulators (16 registers per block) stay live for the whole panel: the
// first 16 sets in AGPRs, the rest in VGPRs through inline asm; the FP64 tile
// (16 BM doubles per lane) is in VGPRs.  The operand fragments of a 16-index
// sub-step (BM blocks of every A slice, one block of every B slice) are held in
// one register set: each is re-read for the next sub-step right after its last
// MFMA in the current one, except those whose last use comes too late for the
// read to land in time (the double-buffered set of t_db), which are read into a
// second buffer at the start of the sub-step.  The two sub-steps of a k-block
// run the products in two orders chosen for that: sub-step 0 walks B's slices
// downward (the A fragments finish late: they are the double-buffered ones),
// sub-step 1 walks A's slices upward.  The k-block's d planes of both operands
// are copied in 1 KB copies, d (BM + 1) per wave, NS k-blocks ahead through a
// ring of NS LDS stages; one barrier per k-block, between its sub-steps.

// Fragment codes: A slice i, block b -> 8 b + i (< 32); B slice j -> 32 + j.
constexpr int fa_code(int i, int b) { return 8 * b + i; }
constexpr int fb_code(int j) { return 32 + j; }
// MFMA t of sub-step order o: code 64 b + 8 i + j (product A_i B_j on block b).
template <int D, int BM>
constexpr int t_mfma(int o, int t) {
    const int npl = D < 6 ? D : 6;
    int n = 0;
    if (o == 1) {
        for (int i = 0; i < npl; ++i)
            for (int b = 0; b < BM; ++b)
                for (int j = 0; j < npl; ++j)
                    if (i + j < D && n++ == t) return 64 * b + 8 * i + j;
    } else {
        for (int j = npl - 1; j >= 0; --j)
            for (int i = 0; i < npl; ++i)
                for (int b = 0; b < BM; ++b)
                    if (i + j < D && n++ == t) return 64 * b + 8 * i + j;
    }
    return -1;
}
template <int D, int BM>
constexpr bool t_uses(int o, int t, int f) {
    const int c = t_mfma<D, BM>(o, t);
    const int b = c >> 6, i = (c >> 3) & 7, j = c & 7;
    return f < 32 ? f == fa_code(i, b) : f == fb_code(j);
}
template <int D, int BM>
constexpr int t_last(int o, int f) {
    int l = -1;
    for (int t = 0; t < n_prod(D) * BM; ++t)
        if (t_uses<D, BM>(o, t, f)) l = t;
    return l;
}
template <int D, int BM>
constexpr int t_first(int o, int f) {
    for (int t = 0; t < n_prod(D) * BM; ++t)
        if (t_uses<D, BM>(o, t, f)) return t;
    return -1;
}
template <int D, int BM>
constexpr bool t_valid(int f) {
    const int npl = D < 6 ? D : 6;
    return f < 32 ? (f % 8 < npl && f / 8 < BM) : f - 32 < npl;
}
// Double-buffered: its last use in sub-step 0 falls in the last W0 MFMAs (the
// read would still be in flight at the barrier that follows), or its last use
// in sub-step 1 in the last W1 (the compiler waits for every outstanding LDS
// read before the first MFMA of a k-block, since the k-block's copies count as
// such events too), or fewer than four MFMAs separate its last use in sub-step
// 1 from its first use in the next sub-step 0.
template <int D, int BM, int W0, int W1>
constexpr bool t_db(int f) {
    const int T = n_prod(D) * BM;
    return t_last<D, BM>(0, f) >= T - W0 || t_last<D, BM>(1, f) >= T - W1 ||
           (T - 1 - t_last<D, BM>(1, f)) + t_first<D, BM>(0, f) < 4;
}
template <int D, int BM, int W0, int W1>
constexpr int t_db_rank(int f) {
    int r = 0;
    for (int g = 0; g < f; ++g)
        if (t_valid<D, BM>(g) && t_db<D, BM, W0, W1>(g)) ++r;
    return r;
}
// Slot after whose MFMA fragment f is read for the next sub-step (order o).
template <int D, int BM, int W0, int W1>
constexpr int t_read_slot(int o, int f) {
    return t_db<D, BM, W0, W1>(f) ? t_db_rank<D, BM, W0, W1>(f) : t_last<D, BM>(o, f);
}
// Product index q of pair (i, j) for d <= 6: diagonal l = i + j ascending, i ascending.
constexpr int q_of(int i, int j) { return (i + j) * (i + j + 1) / 2 + i; }

template <int D, int BM>
struct CfgT {
    static constexpr int P = n_prod(D);
    static constexpr int NPL = D;                                   // d <= 6
    static constexpr int MT = 64 * BM, NT = 64;
    static constexpr int A_BYTES = MT * 64, B_BYTES = NT * 64;      // one plane of a stage
    static constexpr int STAGE = NPL * (A_BYTES + B_BYTES);
    static constexpr int NS = 160 * 1024 / STAGE < 4 ? 160 * 1024 / STAGE : 4;
    static constexpr int COPIES = NPL * (BM + 1);                   // per wave and k-block
    static constexpr int T = P * BM;                                // MFMAs per sub-step
    static constexpr int Q_VGPR = T > 16 ? 16 / BM : P;             // AGPRs hold 16 sets
    static_assert(D >= 3 && D <= 6, "depths 3 .. 6");
    static_assert(4 * COPIES * 1024 == STAGE, "copy split");
    static_assert(NS >= 3 && (NS - 1) * COPIES <= 63, "LDS stages");
};

template <int D, int BM, int W0, int W1>
__global__ __launch_bounds__(256, 1) void gemm_f64t_kernel(
    const uint16_t *__restrict__ Ap, const uint16_t *__restrict__ Bp, double *__restrict__ C,
    int64_t M, int64_t N, int KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
    const int *__restrict__ sa, const int *__restrict__ sb, double alpha, double beta, int nt_m,
    int nt_n) {
    using K = CfgT<D, BM>;
    constexpr int P = K::P, NPL = K::NPL, NS = K::NS, T = K::T;
    __shared__ __attribute__((aligned(1024))) char lds[NS * K::STAGE];

    // groups of 4 tile rows: the 32 tiles resident on an XCD share each A
    // row-panel 8 ways and each B column-panel 4 ways (measured 0.7-3.4 % less
    // GEMM time than groups of 8 at 8192^3, d = 3 .. 6)
    int tm, tn;
    tile_coords<4>(nt_m, nt_n, tm, tn);
    const int lane = threadIdx.x & 63;
    const unsigned lane16 = (unsigned)lane * 16u;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)tm * K::MT, n0 = (int64_t)tn * K::NT;

    // Copy c of a k-block by wave w: for c < NPL BM, part 4 (c % BM) + w (16
    // rows, 1 KB) of A plane c / BM; else part w of B plane c - NPL BM.  ak, bk:
    // the copied k-block's slab of plane 0 at the tile's first row / column.
    const char *Ag = reinterpret_cast<const char *>(Ap) + m0 * 64 + wave * 1024;
    const char *Bg = reinterpret_cast<const char *>(Bp) + n0 * 64 + wave * 1024;
    const int64_t a_plane = plane_elems(KB, RpadA) * 2, b_plane = plane_elems(KB, RpadB) * 2;
    const int64_t a_kstep = RpadA * 64, b_kstep = RpadB * 64;
    auto issue = [&](const char *ak, const char *bk, char *dst, auto c_c) {
        constexpr int c = decltype(c_c)::value;
        if constexpr (c < NPL * BM)
            copy_1k(ak + (c / BM) * a_plane + (c % BM) * 4096,
                    dst + (c / BM) * K::A_BYTES + (c % BM) * 4096 + wave * 1024, lane16);
        else
            copy_1k(bk + (c - NPL * BM) * b_plane,
                    dst + NPL * K::A_BYTES + (c - NPL * BM) * K::B_BYTES + wave * 1024, lane16);
    };
    // copy cursor: the k-block whose copies are issued next (it stays on the
    // last k-block once past it: in bounds, unused) and its stage
    int c_kb = 0, c_st = 0;
    const char *c_ak = Ag, *c_bk = Bg;
    auto cursor_next = [&]() {
        if (c_kb + 1 < KB) {
            ++c_kb;
            c_ak += a_kstep;
            c_bk += b_kstep;
        }
        c_st = c_st + 1 == NS ? 0 : c_st + 1;
    };
    auto stage = [&](int s) -> char * { return lds + s * K::STAGE; };

    const int off0 = frag_offset(lane, 0), off1 = frag_offset(lane, 1);
    const char *const At0 = lds + (wm * 32 * BM) * 64;
    const char *const Bt0 = lds + NPL * K::A_BYTES + (wn * 32) * 64;
    // fragments: [slice][block][buffer]; buffer 1 only for the double-buffered ones
    bf16x8 fa[NPL][BM][2], fb[NPL][2];
    auto read_frag = [&](int so, int off, auto f_c, auto buf_c) {
        constexpr int f = decltype(f_c)::value, u = decltype(buf_c)::value;
        if constexpr (f < 32)
            fa[f % 8][f / 8][u] = lds_frag(At0 + so + (f % 8) * K::A_BYTES + (f / 8) * 32 * 64, off);
        else
            fb[f - 32][u] = lds_frag(Bt0 + so + (f - 32) * K::B_BYTES, off);
    };

    f32x16 acc[P * BM];   // product q, block b at q BM + b
    // Sub-step of order O (= its parity): the T MFMAs, the reads of the next
    // sub-step (stage offset nso, lane offset noff) and NC copies of the
    // cursor's k-block spread over the slots.  MFMA first in every slot: its
    // operands were read a sub-step earlier.
    auto step = [&](auto o_c, auto zero_c, int nso, int noff, auto nc_c) {
        constexpr int O = decltype(o_c)::value;
        constexpr bool zero = decltype(zero_c)::value;
        constexpr int NC = decltype(nc_c)::value;
        char *cdst = stage(c_st);
        static_for<T>([&](auto t_c) {
            constexpr int t = decltype(t_c)::value;
            constexpr int code = t_mfma<D, BM>(O, t), b = code >> 6, i = (code >> 3) & 7,
                          j = code & 7, x = q_of(i, j) * BM + b;
            constexpr int ua = t_db<D, BM, W0, W1>(fa_code(i, b)) ? O : 0;
            constexpr int ub = t_db<D, BM, W0, W1>(fb_code(j)) ? O : 0;
            if constexpr (q_of(i, j) >= K::Q_VGPR) {
                if constexpr (zero) mfma_vacc_zero(acc[x], fa[i][b][ua], fb[j][ub]);
                else mfma_vacc(acc[x], fa[i][b][ua], fb[j][ub]);
            } else {
                acc[x] = mfma(fa[i][b][ua], fb[j][ub], zero ? f32x16{} : acc[x]);
            }
            order_fence();
            static_for<40>([&](auto f_c) {
                constexpr int f = decltype(f_c)::value;
                if constexpr (t_valid<D, BM>(f) && t_read_slot<D, BM, W0, W1>(O, f) == t)
                    read_frag(nso, noff, f_c,
                              std::integral_constant<int, t_db<D, BM, W0, W1>(f) ? 1 - O : 0>{});
            });
            order_fence();
            // NC copies spread over the T slots (the k-th after slot ceil((k + 1) T / NC) - 1)
            if constexpr (NC > 0 && (t * NC) / T != ((t + 1) * NC) / T)
                issue(c_ak, c_bk, cdst, std::integral_constant<int, (t * NC) / T>{});
            order_fence();
        });
    };

    // prologue: k-blocks 0 .. NS - 1 into the stages; wait for k-block 0
    for (int s = 0; s < NS; ++s) {
        static_for<K::COPIES>([&](auto c_c) { issue(c_ak, c_bk, stage(c_st), c_c); });
        cursor_next();
    }
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NS - 1) * K::COPIES) : "memory");
    __syncthreads();
    static_for<40>([&](auto f_c) {
        if constexpr (t_valid<D, BM>(decltype(f_c)::value))
            read_frag(0, off0, f_c, std::integral_constant<int, 0>{});
    });

    double acc64[BM][16];
#pragma unroll
    for (int b = 0; b < BM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc64[b][r] = 0.0;

    int qs = 0;   // stage of the current k-block
    // k-block kb: sub-step 0, wait + barrier, sub-step 1 with the copies of
    // k-block kb + NS (into the stage of kb, which no wave reads any more)
    auto kblock = [&](auto zero_c) {
        const int qn = qs + 1 == NS ? 0 : qs + 1;
        step(std::integral_constant<int, 0>{}, zero_c, qs * K::STAGE, off1,
             std::integral_constant<int, 0>{});
        __builtin_amdgcn_sched_barrier(0);
        // k-block kb + 1 landed: only kb + 2 .. kb + NS - 1 may still be in flight
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"((NS - 2) * K::COPIES) : "memory");
        pipeline_barrier();
        step(std::integral_constant<int, 1>{}, std::false_type{}, qn * K::STAGE, off0,
             std::integral_constant<int, K::COPIES>{});
        __builtin_amdgcn_sched_barrier(0);
        cursor_next();
        qs = qn;
    };
    // whole panels (KB is a multiple of 8: the planes are zero-padded to whole
    // panels, which adds exact zeros to the last panel's sums); the panel's
    // k-blocks are unrolled (a loop over them made the compiler spill the FP64
    // tile around it)
    for (int p0 = 0; p0 < KB; p0 += KB_PER_PANEL) {
        kblock(std::true_type{});
#pragma unroll
        for (int kb = 1; kb < KB_PER_PANEL; ++kb) kblock(std::false_type{});
        // panel end: widen each product exactly and add it in FP64, in order
        // (one product at a time, so that only its values are in flight)
#pragma unroll
        for (int x = K::Q_VGPR * BM; x < P * BM; ++x) mfma_vacc_settle(acc[x]);
        static_for<P>([&](auto q_c) {
            constexpr int q = decltype(q_c)::value;
#pragma unroll
            for (int b = 0; b < BM; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc64[b][r] += (double)acc[q * BM + b][r];
            __builtin_amdgcn_sched_barrier(0);
        });
    }
    // the last trips issued (unused) copies: let them land before the
    // workgroup ends and its LDS is handed to another workgroup
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    const int64_t col = n0 + wn * 32 + (lane & 31);
    const int col_w = (sa != nullptr && col < N) ? sb[col] : 0;
#pragma unroll
    for (int b = 0; b < BM; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = m0 + wm * 32 * BM + b * 32 + acc_row(lane, r);
            if (row < M && col < N) {
                double val = acc64[b][r];
                if (sa != nullptr) val = ldexp(val, sa[row] + col_w);
                C[row * ldc + col] = out_update(val, alpha, beta, C + row * ldc + col);
            }
        }
}

// Blocks per wave of the long-reduction kernel at depth d (0: not used).
// Row blocks per wave: d = 3 takes 128-row tiles like d = 4 (with tiles
// grouped 4 tile-rows per XCD, 5-6 % less time than 192-row tiles at 4096^3 to
// 16384^3).
constexpr int t_bm(int d) { return d == 6 || d == 5 ? 1 : d == 4 || d == 3 ? 2 : 0; }

template <int D, int W0 = 4, int W1 = 8>
hipError_t launch_t64(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M, int64_t N,
                      int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, const int *sa,
                      const int *sb, double alpha, double beta, hipStream_t s) {
    constexpr int BM = t_bm(D);
    using K = CfgT<D, BM>;
    if (KB % KB_PER_PANEL != 0 || RpadA % K::MT != 0 || RpadB % K::NT != 0)
        return hipErrorInvalidValue;
    const int nt_m = (int)((M + K::MT - 1) / K::MT), nt_n = (int)((N + K::NT - 1) / K::NT);
    gemm_f64t_kernel<D, BM, W0, W1><<<nt_m * nt_n, 256, 0, s>>>(
        Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, nt_m, nt_n);
    return hipGetLastError();
}

// Persistent grid of the DGEMM kernels: one workgroup per CU (their LDS use
// allows one), rounded down to a multiple of 8.
int persistent_workgroups() {
    const int cus = device_cu_count();
    return cus < 8 ? 8 : cus / 8 * 8;
}

// PERSIST_OK = false: the caller only launches long reductions here, which
// never take the persistent grid (its instantiation is then not built).
template <int D, int NS, bool ACC64_LDS, int BMW = 1, bool PERSIST_OK = true>
hipError_t launch_w(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M, int64_t N,
                    int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, const int *sa,
                    const int *sb, double alpha, double beta, hipStream_t s) {
    using K = CfgW<D, NS, ACC64_LDS, BMW>;
    const int nt_m = (int)((M + K::MT - 1) / K::MT), nt_n = (int)((N + K::NT - 1) / K::NT);
    const int ntiles = nt_m * nt_n;
    // Short reductions (K <= 1024): one persistent workgroup per CU (a
    // multiple of 8: every workgroup keeps its XCD), so the next tile's first
    // copies overlap a tile's epilogue and store (measured at 16384^2 x 512,
    // d = 6: 17 % less time).  Longer reductions: one workgroup per tile
    // (persistent was 4-9 % slower at K = 8192; a separate instantiation keeps
    // their kernel free of the tile-walking code).  With an odd number of
    // k-blocks a second tile would start on the other fragment buffer, so
    // those always take one tile per workgroup.
    const int pw = persistent_workgroups();
    if constexpr (PERSIST_OK) {
        if (KB % 2 == 0 && KB <= 32 && ntiles > pw) {
            gemm_f64w_kernel<D, NS, ACC64_LDS, true, BMW><<<pw, 256, 0, s>>>(
                Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, nt_m, nt_n,
                ntiles);
            return hipGetLastError();
        }
    }
    gemm_f64w_kernel<D, NS, ACC64_LDS, false, BMW><<<ntiles, 256, 0, s>>>(
        Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, nt_m, nt_n, ntiles);
    return hipGetLastError();
}

template <int D, int BM, int NS, bool ACC64_LDS, int AFTER>
hipError_t launch_t(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M, int64_t N,
                    int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, const int *sa,
                    const int *sb, double alpha, double beta, hipStream_t s) {
    using K = Cfg<D, BM, NS, ACC64_LDS, AFTER>;
    const int nt_m = (int)((M + K::MT - 1) / K::MT), nt_n = (int)((N + K::NT - 1) / K::NT);
    const int ntiles = nt_m * nt_n;
    // short reductions: persistent workgroups (as in launch_w; every k-block
    // starts on f0, so any number of k-blocks works).  A separate
    // instantiation, so that the one-tile kernel of long reductions carries
    // none of the tile-walking code (it cost up to 7 % at 8192 for d = 5).
    const int pw = persistent_workgroups();
    if (KB <= 32 && ntiles > pw)
        gemm_f64_kernel<D, BM, NS, ACC64_LDS, AFTER, true><<<pw, 256, 0, s>>>(
            Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, nt_m, nt_n, ntiles);
    else
        gemm_f64_kernel<D, BM, NS, ACC64_LDS, AFTER, false><<<ntiles, 256, 0, s>>>(
            Ap, Bp, C, M, N, (int)KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, nt_m, nt_n, ntiles);
    return hipGetLastError();
}

}  // namespace

namespace {
// Depths whose long reductions run on gemm_f64t_kernel (whole panels).
constexpr bool T_DEPTH[12] = {false, false, false, true, true, true, true,
                              false, false, false, false, false};

// Whether a depth-d DGEMM of an M x N output with KB k-blocks runs on
// gemm_f64t_kernel: long reductions (K > 1024) whose (64 BM) x 64 tiles fill
// the CUs (smaller grids keep the kernels with smaller tiles).
bool use_t64(int d, int64_t M, int64_t N, int64_t KB) {
    if (d < 3 || d > 6 || !T_DEPTH[d] || KB <= 32) return false;
    const int64_t mt = 64 * t_bm(d);
    return ((M + mt - 1) / mt) * ((N + DGEMM_NT - 1) / DGEMM_NT) >= persistent_workgroups();
}
}  // namespace

int64_t dgemm_tile_rows(int d, int64_t M, int64_t N, int64_t KB) {
    if (use_t64(d, M, N, KB)) return 64 * t_bm(d);
    return d == 1 ? 256 : d <= 3 ? 128 : 64;   // a multiple of every other kernel's tile
}

int64_t dgemm_kb_padded(int d, int64_t M, int64_t N, int64_t KB) {
    return use_t64(d, M, N, KB) ? (KB + KB_PER_PANEL - 1) / KB_PER_PANEL * KB_PER_PANEL : KB;
}

hipError_t launch_gemm_f64(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M,
                           int64_t N, int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
                           const int *sa, const int *sb, double alpha, double beta, int d,
                           hipStream_t s) {
    // Depths 1 .. 5 take the wide kernel's 64 x 64 tiles (BMW = 2) where it
    // measured faster than the 32 x 32 x 16 kernel: long reductions (K > 1024)
    // of d = 2, 4 and 5 (8, 2 and 5 % at 8192^3), and grids of d = 1 .. 3
    // whose 128- or 256-row tiles would number fewer than the CUs (1.5 - 1.9x
    // at 1000 x 1000 x 8200).  The other long reductions of d = 1 take its
    // 128 x 64 tiles (BMW = 4; 7-40 % faster).  Short reductions of d = 1, 2,
    // 4, 5 and the large grids of d = 3 measured faster on the 32 x 32 x 16
    // kernel.  Both kernels give the same bits.
    const int pw = persistent_workgroups();
    auto few_tiles = [&](int64_t mt) {
        return ((M + mt - 1) / mt) * ((N + DGEMM_NT - 1) / DGEMM_NT) < pw;
    };
    const bool long_k = KB > 32;
    if (use_t64(d, M, N, KB)) {
        switch (d) {
            case 3: return launch_t64<3>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            case 4: return launch_t64<4>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            case 5: return launch_t64<5>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            case 6: return launch_t64<6>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            default: return hipErrorInvalidValue;
        }
    }
    switch (d) {
        case 1:
            if (few_tiles(256))
                return launch_w<1, 4, false, 2>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            if (long_k)
                return launch_w<1, 4, false, 4, false>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            return launch_t<1, 4, 4, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 2:
            if (long_k || few_tiles(128))
                return launch_w<2, 4, false, 2>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            return launch_t<2, 2, 4, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 3:
            if (few_tiles(128))
                return launch_w<3, 4, false, 2>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            return launch_t<3, 2, 3, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 4:
            if (long_k)
                return launch_w<4, 4, false, 2, false>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            return launch_t<4, 1, 3, false, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 5:
            if (long_k)
                return launch_w<5, 3, true, 2, false>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
            return launch_t<5, 1, 3, true, 99>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 6: return launch_w<6, 4, false>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 7: return launch_w<7, 3, false>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 8: return launch_w<8, 3, true>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 9: return launch_w<9, 3, true>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 10: return launch_w<10, 3, true>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        case 11: return launch_w<11, 3, true>(Ap, Bp, C, M, N, KB, RpadA, RpadB, ldc, sa, sb, alpha, beta, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace emu
