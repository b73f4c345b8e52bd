// Split/pack kernels: FP32 three-component split (Eq. fp32split, Sec. 4.2) and
// FP64 fixed six-slice simplified Ozaki split (Eq. fp64split, Sec. 4.3), each
// writing BF16 component planes in the packed MFMA operand format described
// in emu_internal.h.  Work item: one 16-byte packed chunk (8 consecutive
// reduction indices of one packed row), so every output store is a 16-byte
// vector store and a wave writes 1 KB contiguously per component.
#include "emu_internal.h"

namespace emu {
namespace {

constexpr int SPLIT_THREADS = 256;
constexpr int ROWS_PER_BLOCK = 64;    // 64 packed rows x 4 chunks = 256 work items

// Zeros that the loads of entries outside an operand read.
__device__ double g_zero8_f64[8];

__device__ inline unsigned block_or(unsigned v) {
    // OR within the wave, then one atomic per wave.
    for (int off = 32; off > 0; off >>= 1) v |= __shfl_xor(v, off);
    return v;
}

// Decode the block's (k-block, row-group) pair and the thread's row/chunk.
struct ItemCoords {
    int64_t kb, prow;
    int q;
};

__device__ inline ItemCoords item_coords(int64_t pair, int RG) {
    ItemCoords c;
    c.kb = pair / RG;
    int64_t rg = pair - c.kb * RG;
    c.prow = rg * ROWS_PER_BLOCK + (threadIdx.x >> 2);
    c.q = threadIdx.x & 3;
    return c;
}

// ---------------------------------------------------------------------------
// FP32: A_r = fl_BF16(A^(r)), A^(r+1) = fl_32(A^(r) - A_r), r = 0, 1, 2.
// AS_B = false: X is rows x cols (an A operand, packed row = X row, k = col).
// AS_B = true : X is rows x cols = K x N (a B operand, packed row = column n,
//               k = X row), i.e. B is packed transposed.
// Blocks [b0, b0 + nb) of the launch serve one operand, block b of them the
// items b, b + nb, ...
template <bool AS_B>
__device__ __forceinline__ void split_f32_operand(const float *__restrict__ X, int64_t rows,
                                                  int64_t cols, int64_t ldx, u16 *__restrict__ P,
                                                  int64_t KB, int64_t Rpad,
                                                  unsigned *__restrict__ status, int b, int nb) {
    const int RG = (int)(Rpad / ROWS_PER_BLOCK);
    const int64_t npairs = KB * RG;
    const int64_t prow_lim = AS_B ? cols : rows;
    const int64_t k_lim = AS_B ? rows : cols;
    unsigned st = 0;
    for (int64_t pair = b; pair < npairs; pair += nb) {
        const ItemCoords ic = item_coords(pair, RG);
        const int64_t k0 = ic.kb * KBLK + ic.q * 8;
        float x[8];
        if (!AS_B) {
            const float *src = X + ic.prow * ldx + k0;
            const bool full = ic.prow < prow_lim && k0 + 8 <= k_lim;
            if (full && ((reinterpret_cast<uintptr_t>(src) & 15u) == 0)) {
                const float4 v0 = *reinterpret_cast<const float4 *>(src);
                const float4 v1 = *reinterpret_cast<const float4 *>(src + 4);
                x[0] = v0.x; x[1] = v0.y; x[2] = v0.z; x[3] = v0.w;
                x[4] = v1.x; x[5] = v1.y; x[6] = v1.z; x[7] = v1.w;
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    x[i] = (ic.prow < prow_lim && k0 + i < k_lim) ? src[i] : 0.0f;
            }
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                x[i] = (ic.prow < prow_lim && k0 + i < k_lim) ? X[(k0 + i) * ldx + ic.prow] : 0.0f;
        }
        u16x8 c0, c1, c2;
        split3_f32x8(x, c0, c1, c2, st);
        *reinterpret_cast<u16x8 *>(P + packed_index(0, ic.kb, ic.prow, ic.q, KB, Rpad)) = c0;
        *reinterpret_cast<u16x8 *>(P + packed_index(1, ic.kb, ic.prow, ic.q, KB, Rpad)) = c1;
        *reinterpret_cast<u16x8 *>(P + packed_index(2, ic.kb, ic.prow, ic.q, KB, Rpad)) = c2;
    }
    st = block_or(st);
    if ((threadIdx.x & 63) == 0 && st) atomicOr(status, st);
}

// Operands of one FP32 split launch (the GEMM splits A and B together).
struct F32SplitArgs {
    F32SplitOperand op[2];
    int nops;
    int blocks0;          // blocks of operand 0; the rest serve operand 1
    int64_t KB;
    unsigned *status;
};

__global__ __launch_bounds__(SPLIT_THREADS) void split_f32_kernel(F32SplitArgs a) {
    const bool second = a.nops > 1 && (int)blockIdx.x >= a.blocks0;
    const F32SplitOperand &op = second ? a.op[1] : a.op[0];
    const int b = (int)blockIdx.x - (second ? a.blocks0 : 0);
    const int nb = second ? (int)gridDim.x - a.blocks0 : a.blocks0;
    if (op.as_b)
        split_f32_operand<true>(op.X, op.rows, op.cols, op.ldx, op.P, a.KB, op.Rpad, a.status, b, nb);
    else
        split_f32_operand<false>(op.X, op.rows, op.cols, op.ldx, op.P, a.KB, op.Rpad, a.status, b, nb);
}

// ---------------------------------------------------------------------------
// FP64 split.  The operand-wide maximum of every level is a global reduction;
// instead of six dependent passes the split speculates the exponent chain
// v_(r+1) = v_r - step (step = 9 for the symmetric projection, 8 for the
// literal one) and records the true maxima of the residuals it produces.  Each
// later pass first verifies the chain against the maxima the previous pass
// recorded, from the first unverified level on; at the first mismatch it
// takes the recorded maximum (exact: every earlier level was computed with
// verified exponents), re-speculates the levels after it and recomputes them.
// Every pass fixes at least one more level, so nlev passes suffice; once the
// chain is verified a pass only copies its state slot forward.  Every block
// runs the (tiny) verification itself from the previous pass's slot, so no
// separate launch is needed between passes.

__device__ inline int ceil_log2_pos(double m) {
    int e;
    const double f = frexp(m, &e);
    return (f == 0.5) ? e - 1 : e;
}

__device__ inline unsigned long long dbits(double x) {
    return (unsigned long long)__double_as_longlong(x);
}

// Operands of one launch and the split of its grid between them.
struct F64SplitArgs {
    F64SplitOperand op[2];
    int nops;
    int blocks0;          // blocks of operand 0; the rest serve operand 1
    int64_t KB;
    unsigned *status;
    int dcheck;           // depth d of the product set to range-check (A = op 0,
                          // B = op 1), or 0 for none
};

// The block's operand (selected, not indexed, so that the arguments stay in the
// kernel-argument segment), its block index and block count within it.
__device__ inline const F64SplitOperand &operand_of_block(const F64SplitArgs &a, int &b, int &nb) {
    const bool second = a.nops > 1 && (int)blockIdx.x >= a.blocks0;
    b = (int)blockIdx.x - (second ? a.blocks0 : 0);
    nb = second ? (int)gridDim.x - a.blocks0 : a.blocks0;
    return second ? a.op[1] : a.op[0];
}

__global__ void f64_state_init(F64SplitArgs a, int nlev, int mode) {
    const int t = threadIdx.x;
    if (t >= a.nops * F64_SLOTS) return;
    F64SplitState &s = a.op[t / F64_SLOTS].st[t % F64_SLOTS];
    for (int r = 0; r < 6; ++r) { s.maxbits[r] = 0ull; s.v[r] = 0; }
    s.replay_from = 0;
    s.nlev = nlev;
    s.mode = mode;
}

// max |x| over an operand (level-0 maximum, into slot 0) and the input-domain
// checks of Eq. (bf16rangefp64).  Rows are strided over the operand's blocks,
// columns over threads.  With weights (sc non-null) the operand is read as
// x 2^-sc[p], p the packed row of x (X's row, or X's column for a B operand),
// and the checks apply to it.
__global__ __launch_bounds__(SPLIT_THREADS) void f64_maxabs_kernel(F64SplitArgs a) {
    __shared__ unsigned long long red[SPLIT_THREADS / 64];
    int b, nb;
    const F64SplitOperand &op = operand_of_block(a, b, nb);
    double m = 0.0;
    unsigned flags = 0;
    const double lo = 0x1p-126, hi = 0x1.fep127;   // (2 - 2^-7) 2^127
    // four independent loads in flight per thread (a row is read in steps of
    // 4 x 256 consecutive entries)
    constexpr int U = 4;
    for (int64_t r = b; r < op.rows; r += nb) {
        const double *row = op.X + r * op.ldx;
        for (int64_t c0 = threadIdx.x; c0 < op.cols; c0 += U * SPLIT_THREADS) {
            double x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t c = c0 + u * SPLIT_THREADS;
                x[u] = c < op.cols ? row[c] : 0.0;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t c = c0 + u * SPLIT_THREADS;
                if (op.sc && c < op.cols) x[u] = ldexp(x[u], -op.sc[op.as_b ? c : r]);
                const double ax = fabs(x[u]);
                if (!__builtin_isfinite(x[u])) { flags |= ST_NAN; continue; }
                if (x[u] != 0.0 && (ax < lo || ax > hi)) flags |= ST_RANGE;
                if (ax > m) m = ax;
            }
        }
    }
    for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
    flags = block_or(flags);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[w] = dbits(m);
        if (flags) atomicOr(a.status, flags);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long bm = red[0];
        for (int i = 1; i < SPLIT_THREADS / 64; ++i) bm = red[i] > bm ? red[i] : bm;
        if (bm) atomicMax(&op.st[0].maxbits[0], bm);
    }
}

// Pass `pass` of the six-slice split of every operand of the launch:
//   Z = fl64(fl64(A^(r) + Sigma) - Sigma), Sigma = c 2^(v_r + 45)
//   (c = 0.75 symmetric, 1 literal), A_r = fl_BF16(Z) (= Z in the domain),
//   A^(r+1) = fl64(A^(r) - A_r); zero slices for a level whose residual is 0.
// Reads slot `pass`, writes slot pass + 1: the chain it used, the first level
// r0 it recomputed (its slices r >= r0 are rewritten) and the maxima
// max|A^(r+1)| of the levels after r0.  nlev <= 6 levels are computed (the
// GEMM never reads slices >= nlev, and they do not influence slices < nlev).
template <bool AS_B>
__device__ __forceinline__ void split_f64_pass(const F64SplitOperand op, int64_t KB, int b, int nb,
                               const int (&v)[6], int r0, int nlev, double cst,
                               F64SplitState *out, unsigned *status) {
    __shared__ unsigned long long red[6][SPLIT_THREADS / 64];
    double sig[6];
    // Levels whose slices are normal BF16 values whenever the chain is right:
    // every Z is a multiple of 2^(v - 8) of magnitude <= 2^v, so for
    // -118 <= v <= 127 a nonzero Z lies in [2^-126, 2^127] and needs at most 8
    // significant bits.  There the BF16 pattern is the top half of (float) Z,
    // the residual is A - Z, and only a non-finite Z (NaN or Inf input) can
    // raise a flag.  Other levels take the general rounding and checks.
    bool plain[6];
#pragma unroll
    for (int r = 0; r < 6; ++r) {
        sig[r] = (v[r] == V_ZERO) ? 0.0 : ldexp(cst, v[r] + 45);
        plain[r] = v[r] != V_ZERO && v[r] >= -118 && v[r] <= 127;
    }
    double mx[6] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    unsigned st = 0;
    const int RG = (int)(op.Rpad / ROWS_PER_BLOCK);
    const int64_t npairs = KB * RG;
    const int64_t prow_lim = AS_B ? op.cols : op.rows;
    const int64_t k_lim = AS_B ? op.rows : op.cols;
    const double *X = op.X;
    const int64_t ldx = op.ldx;
    for (int64_t pair = b; pair < npairs; pair += nb) {
        const ItemCoords ic = item_coords(pair, RG);
        const int64_t k0 = ic.kb * KBLK + ic.q * 8;
        double x[8];
        const int wexp = (op.sc && ic.prow < prow_lim) ? -op.sc[ic.prow] : 0;   // weight 2^-s
        const double *src = X + ic.prow * ldx + k0;
        if (!AS_B && ic.prow < prow_lim && k0 + 8 <= k_lim &&
            (reinterpret_cast<uintptr_t>(src) & 15u) == 0) {
#pragma unroll
            for (int i = 0; i < 8; i += 2) {
                const double2 t = *reinterpret_cast<const double2 *>(src + i);
                x[i] = t.x;
                x[i + 1] = t.y;
            }
        } else {
            // branch-free: an entry outside the operand is read from g_zero8_f64,
            // so the eight loads are issued together
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const bool ok = ic.prow < prow_lim && k0 + i < k_lim;
                const double *e = ok ? X + (AS_B ? (k0 + i) * ldx + ic.prow : ic.prow * ldx + k0 + i)
                                     : g_zero8_f64;
                x[i] = *e;
            }
        }
        if (op.sc) {
#pragma unroll
            for (int i = 0; i < 8; ++i) x[i] = ldexp(x[i], wexp);
        }
        u16x8 outp[6];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            double w = x[i];
#pragma unroll
            for (int r = 0; r < 6; ++r) {
                if (r >= nlev) break;
                u16 h = 0;
                if (plain[r]) {
                    const double t = w + sig[r];
                    const double z = t - sig[r];
                    h = (u16)(__float_as_uint((float)z) >> 16);
                    if ((h & 0x7F80u) == 0x7F80u) st |= ST_OVERFLOW;
                    w = w - z;
                } else if (v[r] != V_ZERO) {
                    const double t = w + sig[r];
                    const double z = t - sig[r];
                    h = bf16_rne_bits((float)z);          // exact for in-domain slices
                    st |= classify(h, z != 0.0);
                    w = w - (double)bf16_to_float(h);
                }
                outp[r][i] = h;
                if (r + 1 < nlev && r >= r0) {
                    const double ax = fabs(w);
                    if (ax > mx[r + 1]) mx[r + 1] = ax;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < 6; ++r)
            if (r >= r0 && r < nlev)
                *reinterpret_cast<u16x8 *>(op.P + packed_index(r, ic.kb, ic.prow, ic.q, KB, op.Rpad)) =
                    outp[r];
    }
    // operand-wide maxima of the recomputed levels
    const int w = threadIdx.x >> 6;
#pragma unroll
    for (int r = 1; r < 6; ++r) {
        double m = mx[r];
        for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
        if ((threadIdx.x & 63) == 0) red[r][w] = dbits(m);
    }
    st = block_or(st);
    if ((threadIdx.x & 63) == 0 && st) atomicOr(status, st);
    __syncthreads();
    if (threadIdx.x < 6 && threadIdx.x >= 1) {
        const int r = threadIdx.x;
        if (r > r0 && r < nlev) {
            unsigned long long bm = red[r][0];
            for (int i = 1; i < SPLIT_THREADS / 64; ++i) bm = red[r][i] > bm ? red[r][i] : bm;
            if (bm) atomicMax(&out->maxbits[r], bm);
        }
    }
}

// The exponent chain pass `pass` uses, from the slot `in` the previous pass
// wrote (slot 0, the level-0 maximum, for pass 0); returns the first level the
// pass recomputes, or -1 once the chain is verified.  Pass p fixes level p for
// good, so the chain of the last pass (nlev - 1) is final for levels < nlev.
__device__ inline int chain_of(const F64SplitState &in, int pass, int step, int (&v)[6]) {
    const int nlev = in.nlev;
    unsigned long long mb[6];
    int r0 = -1;
#pragma unroll
    for (int r = 0; r < 6; ++r) { v[r] = in.v[r]; mb[r] = in.maxbits[r]; }
    if (pass == 0) {
        // speculate the whole chain from the level-0 maximum
        const double m0 = __longlong_as_double((long long)mb[0]);
        const int v0 = (m0 == 0.0) ? V_ZERO : ceil_log2_pos(m0);
#pragma unroll
        for (int r = 0; r < 6; ++r) v[r] = (v0 == V_ZERO) ? V_ZERO : v0 - step * r;
        return 0;
    }
    // verify the levels after the previous pass's first recomputed level
    // (compile-time level indices keep v and mb in registers)
    const int rf = in.replay_from;
    bool done = rf < 0;
#pragma unroll
    for (int r = 1; r < 6; ++r) {
        if (done || r <= rf || r >= nlev) continue;
        if (v[r - 1] == V_ZERO) { v[r] = V_ZERO; continue; }
        const double m = __longlong_as_double((long long)mb[r]);
        if (m == 0.0) {
#pragma unroll
            for (int t = r; t < 6; ++t) v[t] = V_ZERO;
            done = true;
            continue;
        }
        const int vt = ceil_log2_pos(m);
        if (vt == v[r]) continue;
        v[r] = vt;
#pragma unroll
        for (int t = r + 1; t < 6; ++t) v[t] = vt - step * (t - r);
        r0 = r;
        done = true;
    }
    return r0;
}

// Whether every retained panel product is an exact FP32 value for the final
// chains vA, vB.  A slice entry is a multiple of 2^(v - 8) of magnitude at
// most 2^v, so the panel sum of A_i B_j (256 terms) is a multiple of
// u = 2^(vA_i + vB_j - 16) below 2^24 u.  Every partial sum is then a normal
// FP32 value (or 0) when u >= 2^-126 and 2^24 u <= 2^127; outside that range
// the FP32 accumulation may round or overflow.  Pairs with an all-zero slice
// contribute exact zeros.
__device__ inline bool panel_products_in_range(const int (&vA)[6], const int (&vB)[6], int d) {
    bool ok = true;
#pragma unroll
    for (int i = 0; i < 6; ++i)
#pragma unroll
        for (int j = 0; j < 6; ++j) {
            if (i + j >= d || vA[i] == V_ZERO || vB[j] == V_ZERO) continue;
            const int e = vA[i] + vB[j];
            if (e - 16 < -126 || e + 8 > 127) ok = false;
        }
    return ok;
}

__global__ __launch_bounds__(SPLIT_THREADS) void split_f64_kernel(F64SplitArgs a, int pass) {
    int b, nb;
    const F64SplitOperand &op = operand_of_block(a, b, nb);
    const F64SplitState &in = op.st[pass];
    F64SplitState *out = op.st + pass + 1;
    const int nlev = in.nlev, step = in.mode ? 8 : 9;
    int v[6];
    const int r0 = chain_of(in, pass, step, v);
    if (b == 0 && threadIdx.x == 0) {
        // levels <= r0 keep their maxima (all of them once verified); the
        // levels after r0 are filled by this pass's atomics
        for (int r = 0; r < 6; ++r) {
            out->v[r] = v[r];
            if (r0 < 0 || r <= r0) out->maxbits[r] = in.maxbits[r];
        }
        out->replay_from = r0;
        out->nlev = nlev;
        out->mode = in.mode;
        // the last pass holds the final chains: range-check the products
        if (a.dcheck > 0 && pass == nlev - 1 && a.nops == 2 && blockIdx.x == 0) {
            int vb[6];
            (void)chain_of(a.op[1].st[pass], pass, step, vb);
            if (!panel_products_in_range(v, vb, a.dcheck)) atomicOr(a.status, ST_INEXACT);
        }
    }
    if (r0 < 0) return;                                   // verified: nothing to redo
    const double cst = in.mode ? 1.0 : 0.75;
    if (op.as_b) split_f64_pass<true>(op, a.KB, b, nb, v, r0, nlev, cst, out, a.status);
    else split_f64_pass<false>(op, a.KB, b, nb, v, r0, nlev, cst, out, a.status);
}

// ---------------------------------------------------------------------------
// Weights of the scale-aware split: s_p = ceil(log2 max|x|) over each row of X
// (by_col = 0) or each column (by_col = 1), non-finite entries ignored, 0 for
// a row without nonzero entries.  The maxima are reduced as bit patterns of
// non-negative doubles (whose unsigned order is the numeric order).

// one block per row, threads across the row
__global__ __launch_bounds__(SPLIT_THREADS) void row_maxbits_kernel(
    const double *__restrict__ X, int64_t rows, int64_t cols, int64_t ldx,
    unsigned long long *__restrict__ mb) {
    __shared__ unsigned long long red[SPLIT_THREADS / 64];
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
        double m = 0.0;
        for (int64_t c = threadIdx.x; c < cols; c += SPLIT_THREADS) {
            const double x = X[r * ldx + c];
            if (__builtin_isfinite(x)) m = fmax(m, fabs(x));
        }
        for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = dbits(m);
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long b = red[0];
            for (int i = 1; i < SPLIT_THREADS / 64; ++i) b = red[i] > b ? red[i] : b;
            mb[r] = b;
        }
        __syncthreads();
    }
}

// 64 columns per block and a slice of the rows per blockIdx.y; lanes run
// along the columns (coalesced), the four waves over rows; one atomic maximum
// per column and block.  mb must be zero on entry.
__global__ __launch_bounds__(SPLIT_THREADS) void col_maxbits_kernel(
    const double *__restrict__ X, int64_t rows, int64_t cols, int64_t ldx,
    unsigned long long *__restrict__ mb) {
    __shared__ unsigned long long red[SPLIT_THREADS / 64][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t c = (int64_t)blockIdx.x * 64 + lane;
    const int64_t per = (rows + gridDim.y - 1) / gridDim.y;
    const int64_t r0 = (int64_t)blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
    double m = 0.0;
    if (c < cols)
        for (int64_t r = r0 + w; r < r1; r += SPLIT_THREADS / 64) {
            const double x = X[r * ldx + c];
            if (__builtin_isfinite(x)) m = fmax(m, fabs(x));
        }
    red[w][lane] = dbits(m);
    __syncthreads();
    if (w == 0 && c < cols) {
        unsigned long long b = red[0][lane];
        for (int i = 1; i < SPLIT_THREADS / 64; ++i) b = red[i][lane] > b ? red[i][lane] : b;
        if (b) atomicMax(&mb[c], b);
    }
}

__global__ void maxbits_to_exponent_kernel(const unsigned long long *__restrict__ mb, int64_t n,
                                           int *__restrict__ s) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const double m = __longlong_as_double((long long)mb[i]);
        s[i] = (m > 0.0) ? ceil_log2_pos(m) : 0;
    }
}

__global__ void fill_u64_kernel(unsigned long long *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0ull;
}

// Test hook: packed planes back to plain row-major planes in X's orientation.
__global__ void unpack_kernel(const u16 *__restrict__ P, int nc, int64_t KB, int64_t Rpad,
                              int64_t rows, int64_t cols, int as_b, u16 *__restrict__ out) {
    const int64_t total = (int64_t)nc * rows * cols;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t c = i / (rows * cols);
        const int64_t rem = i - c * rows * cols;
        const int64_t r = rem / cols, col = rem - r * cols;
        const int64_t prow = as_b ? col : r;
        const int64_t k = as_b ? r : col;
        const int64_t kb = k / KBLK, q = (k % KBLK) / 8;
        out[i] = P[packed_index((int)c, kb, prow, (int)q, KB, Rpad) + (k % 8)];
    }
}

// The verified chain: the slot written by the last pass.
__global__ void copy_v_kernel(const F64SplitState *st, int32_t *v) {
    if (threadIdx.x < 6) v[threadIdx.x] = st[st[0].nlev].v[threadIdx.x];
}

template <typename T>
__global__ void fill_zero_kernel(T *C, int64_t M, int64_t N, int64_t ldc) {
    for (int64_t r = blockIdx.x; r < M; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < N; c += blockDim.x) C[r * ldc + c] = T(0);
}

int grid_for_pairs(int64_t npairs) {
    const int64_t cap = 8192;
    return (int)(npairs < cap ? (npairs > 0 ? npairs : 1) : cap);
}

// Blocks of an FP64 split pass: about eight work items per block, between
// 1024 and 4096 blocks per operand (fewer blocks also mean fewer atomics on
// the per-level maxima at the end of each block; measured at N = 2048 and
// 8192).
int grid_for_pairs_f64(int64_t npairs) {
    int64_t g = npairs / 8;
    g = g < 1024 ? 1024 : (g > 4096 ? 4096 : g);
    return (int)(npairs < g ? (npairs > 0 ? npairs : 1) : g);
}

}  // namespace

// C = beta C (0 when beta == 0: C is then not read), the BLAS result when
// alpha == 0 or K == 0.
template <typename T>
__global__ void scale_c_kernel(T *C, int64_t M, int64_t N, int64_t ldc, T beta) {
    for (int64_t r = blockIdx.x; r < M; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < N; c += blockDim.x)
            C[r * ldc + c] = (beta == T(0)) ? T(0) : beta * C[r * ldc + c];
}

hipError_t launch_scale_c_f32(float *C, int64_t M, int64_t N, int64_t ldc, float beta,
                              hipStream_t s) {
    const int g = (int)(M < 4096 ? (M > 0 ? M : 1) : 4096);
    scale_c_kernel<float><<<g, 256, 0, s>>>(C, M, N, ldc, beta);
    return hipGetLastError();
}

hipError_t launch_scale_c_f64(double *C, int64_t M, int64_t N, int64_t ldc, double beta,
                              hipStream_t s) {
    const int g = (int)(M < 4096 ? (M > 0 ? M : 1) : 4096);
    scale_c_kernel<double><<<g, 256, 0, s>>>(C, M, N, ldc, beta);
    return hipGetLastError();
}

hipError_t launch_fill_f32(float *C, int64_t M, int64_t N, int64_t ldc, hipStream_t s) {
    const int g = (int)(M < 4096 ? M : 4096);
    fill_zero_kernel<float><<<g, 256, 0, s>>>(C, M, N, ldc);
    return hipGetLastError();
}

hipError_t launch_fill_f64(double *C, int64_t M, int64_t N, int64_t ldc, hipStream_t s) {
    const int g = (int)(M < 4096 ? M : 4096);
    fill_zero_kernel<double><<<g, 256, 0, s>>>(C, M, N, ldc);
    return hipGetLastError();
}

hipError_t launch_split_f32(const F32SplitOperand *ops, int nops, int64_t KB, unsigned *status,
                            hipStream_t s) {
    if (nops < 1 || nops > 2) return hipErrorInvalidValue;
    F32SplitArgs a{};
    for (int o = 0; o < nops; ++o) a.op[o] = ops[o];
    a.nops = nops;
    a.KB = KB;
    a.status = status;
    a.blocks0 = grid_for_pairs(KB * (ops[0].Rpad / ROWS_PER_BLOCK));
    const int g = a.blocks0 + (nops > 1 ? grid_for_pairs(KB * (ops[1].Rpad / ROWS_PER_BLOCK)) : 0);
    split_f32_kernel<<<g, SPLIT_THREADS, 0, s>>>(a);
    return hipGetLastError();
}

// Full FP64 split of the operands: init, level-0 maxima, then nlev passes (the
// first speculative; each later one verifies, and replays only on a mismatch).
hipError_t launch_split_f64(const F64SplitOperand *ops, int nops, int64_t KB, int nlev, int mode,
                            int dcheck, unsigned *status, hipStream_t s) {
    if (nops < 1 || nops > 2 || nlev < 1 || nlev > 6 || (dcheck > 0 && nops != 2))
        return hipErrorInvalidValue;
    F64SplitArgs a{};
    for (int o = 0; o < nops; ++o) a.op[o] = ops[o];
    a.nops = nops;
    a.KB = KB;
    a.status = status;
    a.dcheck = dcheck;
    f64_state_init<<<1, 64, 0, s>>>(a, nlev, mode);
    // at most 512 blocks per operand: each ends in one atomic on the maximum
    auto max_blocks = [](int64_t rows) { return (int)(rows < 512 ? (rows > 0 ? rows : 1) : 512); };
    a.blocks0 = max_blocks(ops[0].rows);
    const int gm = a.blocks0 + (nops > 1 ? max_blocks(ops[1].rows) : 0);
    f64_maxabs_kernel<<<gm, SPLIT_THREADS, 0, s>>>(a);
    a.blocks0 = grid_for_pairs_f64(KB * (ops[0].Rpad / ROWS_PER_BLOCK));
    const int g =
        a.blocks0 + (nops > 1 ? grid_for_pairs_f64(KB * (ops[1].Rpad / ROWS_PER_BLOCK)) : 0);
    for (int pass = 0; pass < nlev; ++pass)
        split_f64_kernel<<<g, SPLIT_THREADS, 0, s>>>(a, pass);
    return hipGetLastError();
}

hipError_t launch_scale_exponents(const double *X, int64_t rows, int64_t cols, int64_t ldx,
                                  bool by_col, unsigned long long *mb, int *sexp, hipStream_t s) {
    const int64_t n = by_col ? cols : rows;
    if (n == 0) return hipSuccess;
    const int fg = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
    if (by_col) {
        fill_u64_kernel<<<fg, 256, 0, s>>>(mb, n);
        const int64_t gx = (cols + 63) / 64;
        int64_t gy = (rows + 255) / 256;                  // about 256 rows per block
        if (gy > 65535) gy = 65535;
        if (gx * gy > 16384) gy = 16384 / gx > 1 ? 16384 / gx : 1;
        col_maxbits_kernel<<<dim3((unsigned)gx, (unsigned)gy), SPLIT_THREADS, 0, s>>>(X, rows, cols,
                                                                                      ldx, mb);
    } else {
        const int g = (int)(rows < 8192 ? rows : 8192);
        row_maxbits_kernel<<<g, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, mb);
    }
    maxbits_to_exponent_kernel<<<fg, 256, 0, s>>>(mb, n, sexp);
    return hipGetLastError();
}

hipError_t launch_unpack(const uint16_t *P, int nc, int64_t KB, int64_t Rpad, int64_t rows,
                         int64_t cols, bool as_b, uint16_t *out, hipStream_t s) {
    unpack_kernel<<<2048, 256, 0, s>>>(P, nc, KB, Rpad, rows, cols, as_b ? 1 : 0, out);
    return hipGetLastError();
}

hipError_t launch_copy_v(const F64SplitState *st, int32_t *v, hipStream_t s) {
    copy_v_kernel<<<1, 64, 0, s>>>(st, v);
    return hipGetLastError();
}

}  // namespace emu
