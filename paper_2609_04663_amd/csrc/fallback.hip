// Native FP64 fallback of the emulated DGEMM (the "fallback handling" the
// paper names for inputs its split cannot represent, Sec. 4.3 and Sec. 9).
//
// fallback_dgemm_kernel recomputes C = alpha op(A) op(B) + beta C in plain
// FP64 (fused multiply-adds on the FP64 matrix cores) when the
// status word of the current call has any domain bit set, and does nothing
// otherwise, so the decision is taken on the device, with no host
// synchronisation: every workgroup reads the word first and returns when it
// is zero.  When it is not, workgroup 0 also adds the call's bits and
// ST_FALLBACK to the accumulated status word.
//
// Tiles: 64 x 64 outputs per workgroup of 256 threads (four waves in a 2 x 2
// grid, 32 x 32 each), on the FP64 matrix cores (v_mfma_f64_16x16x4_f64: each
// wave holds 2 x 2 blocks of 16 x 16 FP64 accumulators).  16-index slabs of
// op(A) and op(B) are staged through LDS, k-major, the next slab's loads in
// flight while the current one is multiplied.
#include "emu_internal.h"
#include "gemm_common.h"

namespace emu {
namespace {

constexpr int FT = 64, FK = 16, FP = FT + 16;   // tile, slab depth, padded LDS row

typedef double f64x4 __attribute__((ext_vector_type(4)));

// The four op(A) and four op(B) entries of the slab at k0 that thread t moves:
// k contiguous in memory -> four consecutive k of one row (column); otherwise
// four consecutive rows (columns) of one k.  Zeros outside the operands.
struct SlabRegs {
    double a[4], b[4];
};

__device__ inline void load_slab(SlabRegs &r, const double *__restrict__ A, int64_t lda, int ta,
                                 const double *__restrict__ B, int64_t ldb, int tb, int64_t M,
                                 int64_t N, int64_t K, int64_t m0, int64_t n0, int64_t k0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        // op(A) entry (m, k)
        const int64_t m = ta ? m0 + (t & 15) * 4 + u : m0 + (t >> 2);
        const int64_t k = ta ? k0 + (t >> 4) : k0 + (t & 3) * 4 + u;
        r.a[u] = (m < M && k < K) ? (ta ? A[k * lda + m] : A[m * lda + k]) : 0.0;
        // op(B) entry (k, n)
        const int64_t kb = tb ? k0 + (t & 3) * 4 + u : k0 + (t >> 4);
        const int64_t n = tb ? n0 + (t >> 2) : n0 + (t & 15) * 4 + u;
        r.b[u] = (kb < K && n < N) ? (tb ? B[n * ldb + kb] : B[kb * ldb + n]) : 0.0;
    }
}

__device__ inline void store_slab(const SlabRegs &r, double (*As)[FP], double (*Bs)[FP], int ta,
                                  int tb) {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        if (ta) As[t >> 4][(t & 15) * 4 + u] = r.a[u];
        else As[(t & 3) * 4 + u][t >> 2] = r.a[u];
        if (tb) Bs[(t & 3) * 4 + u][t >> 2] = r.b[u];
        else Bs[t >> 4][(t & 15) * 4 + u] = r.b[u];
    }
}

__global__ __launch_bounds__(256) void fallback_dgemm_kernel(
    const unsigned *__restrict__ call_status, unsigned *__restrict__ status, int64_t M, int64_t N,
    int64_t K, double alpha, const double *__restrict__ A, int64_t lda, int ta,
    const double *__restrict__ B, int64_t ldb, int tb, double beta, const double *__restrict__ Cin,
    int64_t ldcin, double *__restrict__ C, int64_t ldc) {
    const unsigned flags = *call_status;
    if (flags == 0u) return;
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) atomicOr(status, flags | ST_FALLBACK);
    __shared__ double As[FK][FP];   // As[k][m - m0]
    __shared__ double Bs[FK][FP];   // Bs[k][n - n0]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.y * FT, n0 = (int64_t)blockIdx.x * FT;
    f64x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
    SlabRegs r;
    load_slab(r, A, lda, ta, B, ldb, tb, M, N, K, m0, n0, 0);
    store_slab(r, As, Bs, ta, tb);
    __syncthreads();
    // fragment of a 16 x 4 (A) or 4 x 16 (B) block: lane l holds row (column)
    // l % 16 at k = l / 16 of the 4-index sub-step
    const int fr = lane & 15, fk = lane >> 4;
    for (int64_t k0 = 0; k0 < K; k0 += FK) {
        const bool more = k0 + FK < K;
        if (more) load_slab(r, A, lda, ta, B, ldb, tb, M, N, K, m0, n0, k0 + FK);
#pragma unroll
        for (int ks = 0; ks < FK / 4; ++ks) {
            double a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = As[ks * 4 + fk][wm * 32 + i * 16 + fr];
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = Bs[ks * 4 + fk][wn * 32 + j * 16 + fr];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
        if (more) {
            store_slab(r, As, Bs, ta, tb);
            __syncthreads();
        }
    }
    // block (i, j): lane l holds rows l / 16 + 4 q, column l % 16 (the FP64
    // MFMA's accumulator layout, checked against known products)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 32 + j * 16 + fr;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t m = m0 + wm * 32 + i * 16 + fk + 4 * q;
                if (m < M && n < N)
                    C[m * ldc + n] = out_update(acc[i][j][q], alpha, beta, Cin + m * ldcin + n);
            }
        }
}

__global__ void copy_matrix_f64_kernel(const double *__restrict__ src, int64_t lds,
                                       double *__restrict__ dst, int64_t ldd, int64_t M, int64_t N) {
    for (int64_t r = blockIdx.x; r < M; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < N; c += blockDim.x) dst[r * ldd + c] = src[r * lds + c];
}

}  // namespace

hipError_t launch_fallback_dgemm(const unsigned *call_status, unsigned *status, int64_t M,
                                 int64_t N, int64_t K, double alpha, const double *A, int64_t lda,
                                 bool ta, const double *B, int64_t ldb, bool tb, double beta,
                                 const double *Cin, int64_t ldcin, double *C, int64_t ldc,
                                 hipStream_t s) {
    const dim3 grid((unsigned)((N + FT - 1) / FT), (unsigned)((M + FT - 1) / FT));
    if (grid.y > 65535) return hipErrorInvalidValue;
    fallback_dgemm_kernel<<<grid, 256, 0, s>>>(call_status, status, M, N, K, alpha, A, lda,
                                               ta ? 1 : 0, B, ldb, tb ? 1 : 0, beta, Cin, ldcin, C,
                                               ldc);
    return hipGetLastError();
}

hipError_t launch_copy_matrix_f64(const double *src, int64_t lds, double *dst, int64_t ldd,
                                  int64_t M, int64_t N, hipStream_t s) {
    const int g = (int)(M < 4096 ? M : 4096);
    copy_matrix_f64_kernel<<<g, 256, 0, s>>>(src, lds, dst, ldd, M, N);
    return hipGetLastError();
}

}  // namespace emu
