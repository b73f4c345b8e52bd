// Native FP64 fallback of the emulated DGEMM (the "fallback handling" the
// paper names for inputs its split cannot represent, Sec. 4.3 and Sec. 9).
//
// fallback_dgemm_kernel recomputes C = alpha op(A) op(B) + beta C in plain
// FP64 (fused multiply-adds, ascending k inside each 16-index slab) when the
// status word of the current call has any domain bit set, and does nothing
// otherwise, so the decision is taken on the device, with no host
// synchronisation: every workgroup reads the word first and returns when it
// is zero.  When it is not, workgroup 0 also adds the call's bits and
// ST_FALLBACK to the accumulated status word.
//
// Tiles: 64 x 64 outputs per workgroup of 256 threads, 4 x 4 per thread;
// 16-index slabs of op(A) and op(B) staged through LDS.  A fallback is taken
// for exceptional inputs only, so the kernel favours simplicity over speed.
#include "emu_internal.h"
#include "gemm_common.h"

namespace emu {
namespace {

constexpr int FT = 64, FK = 16;

__global__ __launch_bounds__(256) void fallback_dgemm_kernel(
    const unsigned *__restrict__ call_status, unsigned *__restrict__ status, int64_t M, int64_t N,
    int64_t K, double alpha, const double *__restrict__ A, int64_t lda, int ta,
    const double *__restrict__ B, int64_t ldb, int tb, double beta, const double *__restrict__ Cin,
    int64_t ldcin, double *__restrict__ C, int64_t ldc) {
    const unsigned flags = *call_status;
    if (flags == 0u) return;
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) atomicOr(status, flags | ST_FALLBACK);
    __shared__ double As[FK][FT + 1];
    __shared__ double Bs[FK][FT + 1];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t m0 = (int64_t)blockIdx.y * FT, n0 = (int64_t)blockIdx.x * FT;
    double acc[4][4] = {};
    for (int64_t k0 = 0; k0 < K; k0 += FK) {
        // 1024 entries of each slab, four per thread
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = tid + 256 * u;
            const int r = e / FK, c = e % FK;           // A slab: row r (m), column c (k)
            const int64_t m = m0 + r, k = k0 + c;
            double a = 0.0;
            if (m < M && k < K) a = ta ? A[k * lda + m] : A[m * lda + k];
            As[c][r] = a;
            const int kr = e / FT, nc = e % FT;         // B slab: row kr (k), column nc (n)
            const int64_t kk = k0 + kr, n = n0 + nc;
            double b = 0.0;
            if (kk < K && n < N) b = tb ? B[n * ldb + kk] : B[kk * ldb + n];
            Bs[kr][nc] = b;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FK; ++kk) {
            double a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + ty * 4 + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + tx * 4 + j;
            if (n < N) C[m * ldc + n] = out_update(acc[i][j], alpha, beta, Cin + m * ldcin + n);
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
