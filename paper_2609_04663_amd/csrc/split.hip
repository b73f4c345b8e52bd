// Split/pack kernels: FP32 three-component split (Eq. fp32split, Sec. 4.2) and
// FP64 fixed six-slice simplified Ozaki split (Eq. fp64split, Sec. 4.3), each
// writing BF16 component planes in the packed MFMA operand format described
// in emu_internal.h.  Work item: one 16-byte packed chunk (8 consecutive
// reduction indices of one packed row), so every output store is a 16-byte
// vector store and a wave writes 1 KB contiguously per component.
#include "emu_internal.h"

namespace emu {
namespace {

typedef unsigned short u16;
typedef u16 u16x8 __attribute__((ext_vector_type(8)));

constexpr int SPLIT_THREADS = 256;
constexpr int ROWS_PER_BLOCK = 64;    // 64 packed rows x 4 chunks = 256 work items

// Round a binary32 to BF16, nearest, ties to even, on the bit pattern.
__device__ inline u16 bf16_rne_bits(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u16)((u >> 16) | 0x0040u);   // NaN stays NaN
    return (u16)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ inline float bf16_to_float(u16 h) { return __uint_as_float((uint32_t)h << 16); }

// Status of one stored component: overflow, nonzero subnormal, or underflowed
// to zero from a nonzero source.
__device__ inline unsigned classify(u16 h, bool src_nonzero) {
    unsigned ex = (h >> 7) & 0xFFu, fr = h & 0x7Fu;
    if (ex == 0xFFu) return ST_OVERFLOW;
    if (ex == 0u && (fr != 0u || src_nonzero)) return ST_SUBNORMAL;
    return 0u;
}

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
template <bool AS_B>
__global__ __launch_bounds__(SPLIT_THREADS) void split_f32_kernel(
    const float *__restrict__ X, int64_t rows, int64_t cols, int64_t ldx, u16 *__restrict__ P,
    int64_t KB, int64_t Rpad, unsigned *__restrict__ status) {
    const int RG = (int)(Rpad / ROWS_PER_BLOCK);
    const int64_t npairs = KB * RG;
    const int64_t prow_lim = AS_B ? cols : rows;
    const int64_t k_lim = AS_B ? rows : cols;
    unsigned st = 0;
    for (int64_t pair = blockIdx.x; pair < npairs; pair += gridDim.x) {
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
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float a = x[i];
            const bool fin = __builtin_isfinite(a);
            if (!fin) st |= ST_NAN;
            float r = a;
            const u16 h0 = bf16_rne_bits(r);
            if (fin) st |= classify(h0, r != 0.0f);
            r = r - bf16_to_float(h0);
            const u16 h1 = bf16_rne_bits(r);
            if (fin) st |= classify(h1, r != 0.0f);
            r = r - bf16_to_float(h1);
            const u16 h2 = bf16_rne_bits(r);
            if (fin) st |= classify(h2, r != 0.0f);
            r = r - bf16_to_float(h2);
            if (fin && __builtin_isfinite(r) && r != 0.0f) st |= ST_SUBNORMAL;
            c0[i] = h0; c1[i] = h1; c2[i] = h2;
        }
        *reinterpret_cast<u16x8 *>(P + packed_index(0, ic.kb, ic.prow, ic.q, KB, Rpad)) = c0;
        *reinterpret_cast<u16x8 *>(P + packed_index(1, ic.kb, ic.prow, ic.q, KB, Rpad)) = c1;
        *reinterpret_cast<u16x8 *>(P + packed_index(2, ic.kb, ic.prow, ic.q, KB, Rpad)) = c2;
    }
    st = block_or(st);
    if ((threadIdx.x & 63) == 0 && st) atomicOr(status, st);
}

// ---------------------------------------------------------------------------
// FP64 split state machine.  The operand-wide maximum of every level is a
// global reduction; instead of six dependent passes the split speculates the
// exponent chain v_(r+1) = v_r - step (step = 9 for the symmetric projection,
// 8 for the literal one), records the true maxima of the residuals it
// produces, and a verify step replays from the first level whose recorded
// maximum contradicts the speculation.  Levels before the first mismatch were
// computed with verified exponents, so the recorded maximum at the mismatch is
// the true one; every replay fixes at least one more level.

__device__ inline int ceil_log2_pos(double m) {
    int e;
    const double f = frexp(m, &e);
    return (f == 0.5) ? e - 1 : e;
}

__device__ inline unsigned long long dbits(double x) {
    return (unsigned long long)__double_as_longlong(x);
}

__global__ void f64_state_init(F64SplitState *st, int nst, int nlev, int mode) {
    const int i = threadIdx.x;
    if (i >= nst) return;
    for (int r = 0; r < 6; ++r) { st[i].maxbits[r] = 0ull; st[i].v[r] = 0; }
    st[i].replay_from = 0;
    st[i].nlev = nlev;
    st[i].mode = mode;
}

__global__ void f64_state_speculate(F64SplitState *st, int nst) {
    const int i = threadIdx.x;
    if (i >= nst) return;
    const int step = st[i].mode ? 8 : 9;
    const double m0 = __longlong_as_double((long long)st[i].maxbits[0]);
    const int v0 = (m0 == 0.0) ? V_ZERO : ceil_log2_pos(m0);
    for (int r = 0; r < 6; ++r) {
        st[i].v[r] = (v0 == V_ZERO) ? V_ZERO : v0 - step * r;
        if (r > 0) st[i].maxbits[r] = 0ull;
    }
    st[i].replay_from = 0;
}

__global__ void f64_state_verify(F64SplitState *st, int nst) {
    const int i = threadIdx.x;
    if (i >= nst) return;
    F64SplitState &s = st[i];
    const int step = s.mode ? 8 : 9;
    const int start = s.replay_from < 0 ? s.nlev : s.replay_from + 1;
    s.replay_from = -1;
    for (int r = start; r < s.nlev; ++r) {
        if (s.v[r - 1] == V_ZERO) { s.v[r] = V_ZERO; continue; }
        const double m = __longlong_as_double((long long)s.maxbits[r]);
        if (m == 0.0) {
            for (int t = r; t < 6; ++t) s.v[t] = V_ZERO;
            break;
        }
        const int vt = ceil_log2_pos(m);
        if (vt == s.v[r]) continue;
        s.v[r] = vt;
        for (int t = r + 1; t < 6; ++t) { s.v[t] = vt - step * (t - r); s.maxbits[t] = 0ull; }
        s.replay_from = r;
        break;
    }
}

// max |x| over an operand (level-0 maximum) and the input-domain checks of
// Eq. (bf16rangefp64).  Rows are strided over blocks, columns over threads.
// With weights (sc non-null) the operand is read as x 2^-sc[p], p the packed
// row of x (X's row, or X's column when by_col), and the checks apply to it.
__global__ __launch_bounds__(SPLIT_THREADS) void f64_maxabs_kernel(
    const double *__restrict__ X, int64_t rows, int64_t cols, int64_t ldx,
    const int *__restrict__ sc, int by_col, F64SplitState *__restrict__ st,
    unsigned *__restrict__ status) {
    __shared__ unsigned long long red[SPLIT_THREADS / 64];
    double m = 0.0;
    unsigned flags = 0;
    const double lo = 0x1p-126, hi = 0x1.fep127;   // (2 - 2^-7) 2^127
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
        const double *row = X + r * ldx;
        for (int64_t c = threadIdx.x; c < cols; c += SPLIT_THREADS) {
            double x = row[c];
            if (sc) x = ldexp(x, -sc[by_col ? c : r]);
            const double a = fabs(x);
            if (!__builtin_isfinite(x)) { flags |= ST_NAN; continue; }
            if (x != 0.0 && (a < lo || a > hi)) flags |= ST_RANGE;
            if (a > m) m = a;
        }
    }
    for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
    flags = block_or(flags);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[w] = dbits(m);
        if (flags) atomicOr(status, flags);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long b = red[0];
        for (int i = 1; i < SPLIT_THREADS / 64; ++i) b = red[i] > b ? red[i] : b;
        if (b) atomicMax(&st->maxbits[0], b);
    }
}

// One speculative (first_pass) or replay pass of the six-slice split:
//   Z = fl64(fl64(A^(r) + Sigma) - Sigma), Sigma = c 2^(v_r + 45)
//   (c = 0.75 symmetric, 1 literal), A_r = fl_BF16(Z) (= Z in the domain),
//   A^(r+1) = fl64(A^(r) - A_r); zero slices for a level whose residual is 0.
// Writes slices r >= first recomputed level, records max|A^(r+1)| of the
// levels after it.  nlev <= 6 levels are computed (the GEMM never reads
// slices >= d, and they do not influence slices < d).
template <bool AS_B>
__global__ __launch_bounds__(SPLIT_THREADS) void split_f64_kernel(
    const double *__restrict__ X, int64_t rows, int64_t cols, int64_t ldx,
    const int *__restrict__ sc, u16 *__restrict__ P, int64_t KB, int64_t Rpad,
    F64SplitState *__restrict__ stp, unsigned *__restrict__ status, int first_pass) {
    __shared__ unsigned long long red[6][SPLIT_THREADS / 64];
    const int r0 = first_pass ? 0 : stp->replay_from;
    if (r0 < 0) return;                                   // verified: nothing to redo
    const int nlev = stp->nlev;
    int v[6];
    double sig[6];
    const double cst = stp->mode ? 1.0 : 0.75;
#pragma unroll
    for (int r = 0; r < 6; ++r) {
        v[r] = stp->v[r];
        sig[r] = (v[r] == V_ZERO) ? 0.0 : ldexp(cst, v[r] + 45);
    }
    double mx[6] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    unsigned st = 0;
    const int RG = (int)(Rpad / ROWS_PER_BLOCK);
    const int64_t npairs = KB * RG;
    const int64_t prow_lim = AS_B ? cols : rows;
    const int64_t k_lim = AS_B ? rows : cols;
    for (int64_t pair = blockIdx.x; pair < npairs; pair += gridDim.x) {
        const ItemCoords ic = item_coords(pair, RG);
        const int64_t k0 = ic.kb * KBLK + ic.q * 8;
        double x[8];
        const int wexp = (sc && ic.prow < prow_lim) ? -sc[ic.prow] : 0;   // row weight 2^-s
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const bool ok = ic.prow < prow_lim && k0 + i < k_lim;
            x[i] = ok ? (AS_B ? X[(k0 + i) * ldx + ic.prow] : X[ic.prow * ldx + k0 + i]) : 0.0;
            if (sc) x[i] = ldexp(x[i], wexp);
        }
        u16x8 out[6];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            double w = x[i];
#pragma unroll
            for (int r = 0; r < 6; ++r) {
                if (r >= nlev) break;
                u16 h = 0;
                if (v[r] != V_ZERO) {
                    const double t = w + sig[r];
                    const double z = t - sig[r];
                    h = bf16_rne_bits((float)z);          // exact for in-domain slices
                    st |= classify(h, z != 0.0);
                    w = w - (double)bf16_to_float(h);
                }
                out[r][i] = h;
                if (r + 1 < nlev && r >= r0) {
                    const double a = fabs(w);
                    if (a > mx[r + 1]) mx[r + 1] = a;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < 6; ++r)
            if (r >= r0 && r < nlev)
                *reinterpret_cast<u16x8 *>(P + packed_index(r, ic.kb, ic.prow, ic.q, KB, Rpad)) =
                    out[r];
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
            unsigned long long b = red[r][0];
            for (int i = 1; i < SPLIT_THREADS / 64; ++i) b = red[r][i] > b ? red[r][i] : b;
            if (b) atomicMax(&stp->maxbits[r], b);
        }
    }
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

__global__ void copy_v_kernel(const F64SplitState *st, int32_t *v) {
    if (threadIdx.x < 6) v[threadIdx.x] = st->v[threadIdx.x];
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

hipError_t launch_split_f32(const float *X, int64_t rows, int64_t cols, int64_t ldx, bool as_b,
                            uint16_t *P, int64_t KB, int64_t Rpad, unsigned *status,
                            hipStream_t s) {
    const int g = grid_for_pairs(KB * (Rpad / ROWS_PER_BLOCK));
    if (as_b)
        split_f32_kernel<true><<<g, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, P, KB, Rpad, status);
    else
        split_f32_kernel<false><<<g, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, P, KB, Rpad, status);
    return hipGetLastError();
}

// Full FP64 split of one operand: init, level-0 maximum, speculative pass,
// then verify/replay until every level is verified (at most nlev - 1 replays,
// each a no-op once the chain is verified), then a final verify.
hipError_t launch_split_f64(const double *X, int64_t rows, int64_t cols, int64_t ldx, bool as_b,
                            const int *sc, uint16_t *P, int64_t KB, int64_t Rpad, int nlev,
                            int mode, F64SplitState *st, unsigned *status, hipStream_t s) {
    f64_state_init<<<1, 64, 0, s>>>(st, 1, nlev, mode);
    const int gm = (int)(rows < 2048 ? (rows > 0 ? rows : 1) : 2048);
    f64_maxabs_kernel<<<gm, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, sc, as_b ? 1 : 0, st, status);
    f64_state_speculate<<<1, 64, 0, s>>>(st, 1);
    const int g = grid_for_pairs(KB * (Rpad / ROWS_PER_BLOCK));
    for (int pass = 0; pass < nlev; ++pass) {
        if (pass > 0) f64_state_verify<<<1, 64, 0, s>>>(st, 1);
        if (as_b)
            split_f64_kernel<true><<<g, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, sc, P, KB, Rpad,
                                                                st, status, pass == 0);
        else
            split_f64_kernel<false><<<g, SPLIT_THREADS, 0, s>>>(X, rows, cols, ldx, sc, P, KB, Rpad,
                                                                 st, status, pass == 0);
    }
    f64_state_verify<<<1, 64, 0, s>>>(st, 1);
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
