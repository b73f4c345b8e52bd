// K-binned scale-aware scope (EMU_SCOPE_KBIN): classes of the reduction
// indices and the gathers of the index groups.  An extension of the
// scale-aware decomposition the paper names as its key next step (Sec. 9)
// along the reduction: the products a_mk b_kn of one k share the magnitude
// class of k, the indices of one class form a group, and every group is
// emulated with its own row/column weights and exponent chains.
//
// class(k) = min(NCLS - 1, floor(-(ceil(log2 max_m |a~_mk|) +
//                                  ceil(log2 max_n |b~_kn|)) / WIDTH)),
// a~ = op(A) with row m scaled by 2^-sA_m, b~ = op(B) with column n scaled by
// 2^-sB_n (the ROWCOL weights); -1 when either maximum is 0 (the index
// contributes exact zeros and is left out).
#include "emu_internal.h"

namespace emu {
namespace {

constexpr int KT = 256;

__device__ inline unsigned long long mbits(double x) {
    return (unsigned long long)__double_as_longlong(x);
}

// mb[k] = max over the other index of |X| 2^-w (finite entries), X stored
// rows x cols (ldx); k runs along the columns (k_is_col) or the rows, and w is
// indexed by the other coordinate.  One atomic maximum per k and block; mb
// must be zero on entry.
__global__ __launch_bounds__(KT) void weighted_kmax_kernel(const double *__restrict__ X,
                                                           int64_t rows, int64_t cols, int64_t ldx,
                                                           int k_is_col, const int *__restrict__ w,
                                                           unsigned long long *__restrict__ mb) {
    if (k_is_col) {
        // lanes along the columns (coalesced), the block's rows strided
        const int64_t c = (int64_t)blockIdx.x * KT + threadIdx.x;
        if (c >= cols) return;
        const int64_t per = (rows + gridDim.y - 1) / gridDim.y;
        const int64_t r0 = (int64_t)blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
        double m = 0.0;
        for (int64_t r = r0; r < r1; ++r) {
            const double x = X[r * ldx + c];
            if (__builtin_isfinite(x)) m = fmax(m, fabs(ldexp(x, -w[r])));
        }
        if (m > 0.0) atomicMax(&mb[c], mbits(m));
    } else {
        // one row per block iteration, threads along it
        __shared__ unsigned long long red[KT / 64];
        for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
            double m = 0.0;
            for (int64_t c = threadIdx.x; c < cols; c += KT) {
                const double x = X[r * ldx + c];
                if (__builtin_isfinite(x)) m = fmax(m, fabs(ldexp(x, -w[c])));
            }
            for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
            if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mbits(m);
            __syncthreads();
            if (threadIdx.x == 0) {
                unsigned long long b = red[0];
                for (int i = 1; i < KT / 64; ++i) b = red[i] > b ? red[i] : b;
                if (b) atomicMax(&mb[r], b);
            }
            __syncthreads();
        }
    }
}

__device__ inline int ceil_log2_d(double m) {
    int e;
    const double f = frexp(m, &e);
    return (f == 0.5) ? e - 1 : e;
}

__global__ void kclass_kernel(const unsigned long long *__restrict__ ma,
                              const unsigned long long *__restrict__ mb, int64_t K, int width,
                              int ncls, int *__restrict__ cls) {
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < K;
         k += (int64_t)gridDim.x * blockDim.x) {
        const double a = __longlong_as_double((long long)ma[k]);
        const double b = __longlong_as_double((long long)mb[k]);
        int c = -1;
        if (a > 0.0 && b > 0.0) {
            const int ne = -(ceil_log2_d(a) + ceil_log2_d(b));   // >= 0: a, b <= 1
            c = ne / width < ncls - 1 ? ne / width : ncls - 1;
        }
        cls[k] = c;
    }
}

__global__ void fill_u64_zero_kernel(unsigned long long *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0ull;
}

// Columns idx[0 .. kb) of op(A) (A stored M x K, or K x M when ta) into a
// row-major M x kb matrix G.
__global__ void gather_opa_kernel(const double *__restrict__ A, int64_t lda, int ta, int64_t M,
                                  const int *__restrict__ idx, int64_t kb, double *__restrict__ G) {
    for (int64_t m = blockIdx.x; m < M; m += gridDim.x)
        for (int64_t j = threadIdx.x; j < kb; j += blockDim.x) {
            const int64_t k = idx[j];
            G[m * kb + j] = ta ? A[k * lda + m] : A[m * lda + k];
        }
}

// Rows idx[0 .. kb) of op(B) (B stored K x N, or N x K when tb) into a
// row-major kb x N matrix G.
__global__ void gather_opb_kernel(const double *__restrict__ B, int64_t ldb, int tb, int64_t N,
                                  const int *__restrict__ idx, int64_t kb, double *__restrict__ G) {
    for (int64_t j = blockIdx.x; j < kb; j += gridDim.x) {
        const int64_t k = idx[j];
        for (int64_t n = threadIdx.x; n < N; n += blockDim.x)
            G[j * N + n] = tb ? B[n * ldb + k] : B[k * ldb + n];
    }
}

// C = fl(fl(alpha P) + fl(beta C)) (fl(alpha P) when beta == 0), unless the
// call's status word says that the fallback has written C already.
__global__ void axpby_f64_kernel(const double *__restrict__ P, int64_t ldp, double *__restrict__ C,
                                 int64_t ldc, int64_t M, int64_t N, double alpha, double beta,
                                 const unsigned *__restrict__ skip_if) {
    if (skip_if != nullptr && *skip_if != 0u) return;
    for (int64_t r = blockIdx.x; r < M; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < N; c += blockDim.x) {
#pragma clang fp contract(off)
            const double ap = alpha * P[r * ldp + c];
            C[r * ldc + c] = beta == 0.0 ? ap : ap + beta * C[r * ldc + c];
        }
}

int grid_rows(int64_t n) { return (int)(n < 4096 ? (n > 0 ? n : 1) : 4096); }

}  // namespace

hipError_t launch_kbin_classes(const double *A, int64_t lda, bool ta, const double *B, int64_t ldb,
                               bool tb, int64_t M, int64_t N, int64_t K, const int *sa,
                               const int *sb, unsigned long long *ma, unsigned long long *mb,
                               int width, int ncls, int *cls, hipStream_t s) {
    const int fg = (int)((2 * K + 255) / 256 < 1024 ? (2 * K + 255) / 256 : 1024);
    fill_u64_zero_kernel<<<fg, 256, 0, s>>>(ma, K);
    fill_u64_zero_kernel<<<fg, 256, 0, s>>>(mb, K);
    // op(A): k along A's columns (stored M x K) or rows (stored K x M); weights sa by m
    auto launch = [&](const double *X, int64_t rows, int64_t cols, int64_t ld, bool k_is_col,
                      const int *w, unsigned long long *out) {
        if (k_is_col) {
            const int64_t gx = (cols + KT - 1) / KT;
            int64_t gy = (rows + 255) / 256;
            if (gy > 65535) gy = 65535;
            if (gx * gy > 16384) gy = 16384 / gx > 1 ? 16384 / gx : 1;
            weighted_kmax_kernel<<<dim3((unsigned)gx, (unsigned)gy), KT, 0, s>>>(X, rows, cols, ld,
                                                                                  1, w, out);
        } else {
            weighted_kmax_kernel<<<grid_rows(rows), KT, 0, s>>>(X, rows, cols, ld, 0, w, out);
        }
    };
    if (ta) launch(A, K, M, lda, false, sa, ma);
    else launch(A, M, K, lda, true, sa, ma);
    // op(B): k along B's rows (stored K x N) or columns (stored N x K); weights sb by n
    if (tb) launch(B, N, K, ldb, true, sb, mb);
    else launch(B, K, N, ldb, false, sb, mb);
    kclass_kernel<<<fg, 256, 0, s>>>(ma, mb, K, width, ncls, cls);
    return hipGetLastError();
}

hipError_t launch_kbin_gather(const double *A, int64_t lda, bool ta, const double *B, int64_t ldb,
                              bool tb, int64_t M, int64_t N, const int *idx, int64_t kb,
                              double *GA, double *GB, hipStream_t s) {
    gather_opa_kernel<<<grid_rows(M), 256, 0, s>>>(A, lda, ta ? 1 : 0, M, idx, kb, GA);
    gather_opb_kernel<<<grid_rows(kb), 256, 0, s>>>(B, ldb, tb ? 1 : 0, N, idx, kb, GB);
    return hipGetLastError();
}

hipError_t launch_axpby_f64(const double *P, int64_t ldp, double *C, int64_t ldc, int64_t M,
                            int64_t N, double alpha, double beta, const unsigned *skip_if,
                            hipStream_t s) {
    axpby_f64_kernel<<<grid_rows(M), 256, 0, s>>>(P, ldp, C, ldc, M, N, alpha, beta, skip_if);
    return hipGetLastError();
}

}  // namespace emu
