// Internal definitions shared by the HIP kernels and the host library.
//
// Packed operand format (the bf16 MFMA operand layout written by the split
// kernels and read by the GEMM kernels).  An operand is viewed as R "rows" by
// K reduction indices: for A the rows are A's rows; for B (K x N) the rows are
// B's columns, i.e. B is stored transposed so that every row is K-contiguous.
//
//   element (c, row, k) of component plane c lives at bf16 index
//     c * plane_elems(KB, Rpad) + (kb * Rpad + row) * 32 + 8 * (q ^ swz(row)) + (k % 8)
//   with kb = k / 32, q = (k % 32) / 8, swz(row) = (row >> 2) & 3,
//   KB = ceil(K / 32) (or more: zero k-blocks), Rpad = R rounded up to a
//   multiple of 64 and of the GEMM tile extent along the rows (plus
//   ROW_SKEW_TILES tiles), plane_elems = KB * Rpad * 32 + PLANE_SKEW.
//
// So one k-block of a component is a row-major [Rpad][32] bf16 slab, 64 bytes
// per row: a workgroup tile of T rows is one contiguous T*64-byte block that a
// direct global->LDS copy moves as is.  The 16-byte chunks inside a row are
// XOR-swizzled by bits 2..3 of the row: an MFMA operand read (ds_read_b128,
// lane l reads one 16-byte chunk of row l % 32) then touches 16 distinct
// 16-byte bank groups in every group of 16 lanes, which the gfx950 LDS (64
// banks) serves without conflict (measured: 164 B/clk/CU, against 111 for
// bits 1..2 and 61 unswizzled).  Padding rows and k >= K are zero.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace emu {

constexpr int KBLK = 32;        // reduction indices per k-block (one LDS stage)
constexpr int ROW_GROUP = 64;   // packed rows are padded to a multiple of this ...
constexpr int KPANEL = 256;     // reduction panel B_K of the FP32/FP64 reconstruction

// ... and of the GEMM tile that reads them (output tile rows for A, columns for B).
constexpr int SGEMM_NT = 128;   // SGEMM output tiles: (192 or 128) x 128
constexpr int DGEMM_NT = 64;
// Slices of each operand that the products of depth d read (indices < 6).
inline int dgemm_planes(int d) { return d < 6 ? d : 6; }
constexpr int KB_PER_PANEL = KPANEL / KBLK;

__host__ __device__ inline int swz(int64_t row) { return (int)((row >> 2) & 3); }

// Memory-channel staggering of the packed operands.  With power-of-two sizes
// the k-block stride (Rpad x 64 B) and the plane stride are multiples of a
// large power of two, and every copy of a tile's k-block (all planes) lands in
// the same few L2 channels.  Two skews break that: Rpad gets ROW_SKEW_TILES
// extra (zero) tiles, and consecutive planes are PLANE_SKEW elements further
// apart than their KB x Rpad x 32 elements (a multiple of 512: planes stay
// 1 KB aligned).
constexpr int ROW_SKEW_TILES = 2;
constexpr int64_t PLANE_SKEW = 2048;

// Elements from one component plane to the next.
__host__ __device__ inline int64_t plane_elems(int64_t KB, int64_t Rpad) {
    return KB * Rpad * KBLK + PLANE_SKEW;
}

__host__ __device__ inline int64_t packed_index(int c, int64_t kb, int64_t row, int q, int64_t KB,
                                                int64_t Rpad) {
    return c * plane_elems(KB, Rpad) + (kb * Rpad + row) * KBLK + 8 * (q ^ swz(row));
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Status bits (same values as EMU_STATUS_* in emu.h).
constexpr unsigned ST_NAN = 1u, ST_RANGE = 2u, ST_SUBNORMAL = 4u, ST_OVERFLOW = 8u, ST_INEXACT = 16u,
                   ST_FALLBACK = 32u;

// Device state of the FP64 split of one operand: the operand-wide per-level
// maxima (bit patterns of non-negative doubles, whose unsigned order is the
// numeric order), the exponent chain v, and the first level the pass that
// wrote it recomputed (-1 once the chain is verified).  One slot per pass:
// slot 0 holds the level-0 maximum, slot p + 1 the state after pass p, so a
// pass only reads a slot that an earlier launch completed.
struct alignas(64) F64SplitState {
    unsigned long long maxbits[6];
    int v[6];
    int replay_from;
    int nlev;
    int mode;
    int pad[3];
};
constexpr int F64_SLOTS = 7;    // nlev <= 6 passes

// One operand of an FP32 split launch.
struct F32SplitOperand {
    const float *X;
    int64_t rows, cols, ldx;    // X as stored
    int as_b;                   // packed rows are X's columns (a B operand)
    uint16_t *P;                // packed planes
    int64_t Rpad;
};

// One operand of an FP64 split launch (the GEMM splits A and B in one launch
// per phase).
struct F64SplitOperand {
    const double *X;
    int64_t rows, cols, ldx;    // X as stored
    int as_b;                   // packed rows are X's columns (a B operand)
    const int *sc;              // per-packed-row weights 2^-sc (scale-aware split) or null
    uint16_t *P;                // packed planes
    int64_t Rpad;
    F64SplitState *st;          // F64_SLOTS slots
};

constexpr int V_ZERO = (int)0x80000000;   // level whose residual is identically zero

typedef unsigned short u16;
typedef u16 u16x8 __attribute__((ext_vector_type(8)));

// Round a binary32 to BF16, nearest, ties to even, on the bit pattern (a NaN
// stays a NaN).  Written with selects, not branches: the streamed-split GEMM
// runs it between its matrix instructions.
__device__ inline u16 bf16_rne_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t rne = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    const uint32_t nan = (u >> 16) | 0x0040u;
    return (u16)(((u & 0x7FFFFFFFu) > 0x7F800000u) ? nan : rne);
}

__device__ inline float bf16_to_float(u16 h) { return __uint_as_float((uint32_t)h << 16); }

// Status of one stored component: overflow, nonzero subnormal, or underflowed
// to zero from a nonzero source.
__device__ inline unsigned classify(u16 h, bool src_nonzero) {
    const unsigned ex = (h >> 7) & 0xFFu, fr = h & 0x7Fu;
    return (ex == 0xFFu ? ST_OVERFLOW : 0u) |
           ((ex == 0u && (fr != 0u || src_nonzero)) ? ST_SUBNORMAL : 0u);
}

// The three BF16 components of an FP32 value (Eq. fp32split, Sec. 4.2):
// A_r = fl_BF16(A^(r)), A^(r+1) = fl_32(A^(r) - A_r), r = 0, 1, 2, with the
// input-domain status bits (a non-finite input; a component that overflows,
// is subnormal or underflows; a nonzero residual after the third).  The split
// kernel and the streamed-split SGEMM both use it.
__device__ inline void split3_f32(float a, u16 &c0, u16 &c1, u16 &c2, unsigned &st) {
    {
        const bool fin = __builtin_isfinite(a);
        float r = a;
        const u16 h0 = bf16_rne_bits(r);
        unsigned f = classify(h0, r != 0.0f);
        r = r - bf16_to_float(h0);
        const u16 h1 = bf16_rne_bits(r);
        f |= classify(h1, r != 0.0f);
        r = r - bf16_to_float(h1);
        const u16 h2 = bf16_rne_bits(r);
        f |= classify(h2, r != 0.0f);
        r = r - bf16_to_float(h2);
        f |= (__builtin_isfinite(r) && r != 0.0f) ? ST_SUBNORMAL : 0u;
        st |= fin ? f : ST_NAN;
        c0 = h0;
        c1 = h1;
        c2 = h2;
    }
}
__device__ inline void split3_f32x8(const float (&x)[8], u16x8 &c0, u16x8 &c1, u16x8 &c2,
                                    unsigned &st) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        u16 h0, h1, h2;
        split3_f32(x[i], h0, h1, h2, st);
        c0[i] = h0;
        c1[i] = h1;
        c2[i] = h2;
    }
}

}  // namespace emu

// Launch wrappers (defined in the .hip files, called by the host API).
namespace emu {
hipError_t launch_fill_f32(float *C, int64_t M, int64_t N, int64_t ldc, hipStream_t s);
hipError_t launch_fill_f64(double *C, int64_t M, int64_t N, int64_t ldc, hipStream_t s);
hipError_t launch_scale_c_f32(float *C, int64_t M, int64_t N, int64_t ldc, float beta,
                              hipStream_t s);
hipError_t launch_scale_c_f64(double *C, int64_t M, int64_t N, int64_t ldc, double beta,
                              hipStream_t s);
// The FP32 split of nops <= 2 operands with the same KB, one launch.
hipError_t launch_split_f32(const F32SplitOperand *ops, int nops, int64_t KB, unsigned *status,
                            hipStream_t s);
// The FP64 split of nops <= 2 operands with the same KB: nlev <= 6 levels
// (planes) each, 2 + nlev launches in all.  dcheck = d > 0 (with nops = 2, A
// then B): also set ST_INEXACT when a product of S_d may leave FP32's exact
// range.
hipError_t launch_split_f64(const F64SplitOperand *ops, int nops, int64_t KB, int nlev, int mode,
                            int dcheck, unsigned *status, hipStream_t s);
// per-row (by_col = 0) or per-column exponents ceil(log2 max|x|) of X; mb is
// scratch of rows (or cols) 64-bit words
hipError_t launch_scale_exponents(const double *X, int64_t rows, int64_t cols, int64_t ldx,
                                  bool by_col, unsigned long long *mb, int *sexp, hipStream_t s);
hipError_t launch_unpack(const uint16_t *P, int nc, int64_t KB, int64_t Rpad, int64_t rows,
                         int64_t cols, bool as_b, uint16_t *out, hipStream_t s);
hipError_t launch_copy_v(const F64SplitState *st, int32_t *v, hipStream_t s);
// Native FP64 fallback: C = alpha op(A) op(B) + beta Cin when *call_status is
// nonzero (then also status |= *call_status | ST_FALLBACK); nothing otherwise.
hipError_t launch_fallback_dgemm(const unsigned *call_status, unsigned *status, int64_t M,
                                 int64_t N, int64_t K, double alpha, const double *A, int64_t lda,
                                 bool ta, const double *B, int64_t ldb, bool tb, double beta,
                                 const double *Cin, int64_t ldcin, double *C, int64_t ldc,
                                 hipStream_t s);
hipError_t launch_copy_matrix_f64(const double *src, int64_t lds, double *dst, int64_t ldd,
                                  int64_t M, int64_t N, hipStream_t s);
// K-binned scope: the class of every reduction index of op(A) op(B) (-1: left
// out) from the ROWCOL weights sa, sb; ma, mb: K 64-bit words of scratch each.
constexpr int KBIN_WIDTH = 8, KBIN_MAX = 8;
hipError_t launch_kbin_classes(const double *A, int64_t lda, bool ta, const double *B, int64_t ldb,
                               bool tb, int64_t M, int64_t N, int64_t K, const int *sa,
                               const int *sb, unsigned long long *ma, unsigned long long *mb,
                               int width, int ncls, int *cls, hipStream_t s);
// op(A)'s columns and op(B)'s rows idx[0 .. kb) into row-major M x kb and kb x N
hipError_t launch_kbin_gather(const double *A, int64_t lda, bool ta, const double *B, int64_t ldb,
                              bool tb, int64_t M, int64_t N, const int *idx, int64_t kb,
                              double *GA, double *GB, hipStream_t s);
// C = alpha P + beta C (the BLAS update), skipped when *skip_if is nonzero
hipError_t launch_axpby_f64(const double *P, int64_t ldp, double *C, int64_t ldc, int64_t M,
                            int64_t N, double alpha, double beta, const unsigned *skip_if,
                            hipStream_t s);
// alpha, beta: C = alpha P + beta C (see out_update); 1, 0 stores P
// Split-K factor of the emulated SGEMM: 1 unless the output tiles fill at most
// half of the chip, else up to 16 splits of whole reduction panels.  splits > 1 needs part:
// splits x M x N floats of scratch for the partial sums.
// CUs of the current device (256 on MI355X), read once per process.
int device_cu_count();
int sgemm_tile_m(int64_t M, int64_t N, int64_t KB);   // 192 or 128 output rows per tile
int sgemm_splits(int64_t M, int64_t N, int64_t KB, int tile_m);
// The streamed-split SGEMM: op(A) op(B) read in FP32 by the GEMM, split per
// k-block in the workgroup (128 x 128 tiles); same result bits as the split
// kernel followed by launch_gemm_f32 with 128-row tiles and the same splits.
hipError_t launch_gemm_f32_streamed(const float *A, int64_t lda, bool ta, const float *B,
                                    int64_t ldb, bool tb, float *C, int64_t M, int64_t N,
                                    int64_t K, int64_t ldc, float alpha, float beta, int splits,
                                    float *part, unsigned *status, hipStream_t s);
hipError_t launch_gemm_f32(const uint16_t *Ap, const uint16_t *Bp, float *C, int64_t M, int64_t N,
                           int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc, float alpha,
                           float beta, int tile_m, int splits, float *part, hipStream_t s);
// Packed layout of a depth-d DGEMM (M x N output, KB k-blocks of data) for the
// kernel that will run it: A's rows are padded to a multiple of
// dgemm_tile_rows (B's columns to DGEMM_NT), and the reduction to
// dgemm_kb_padded k-blocks (some kernels run whole panels; the padding is zero).
int64_t dgemm_tile_rows(int d, int64_t M, int64_t N, int64_t KB);
int64_t dgemm_kb_padded(int d, int64_t M, int64_t N, int64_t KB);
// sa, sb: row weights of A and column weights of B to restore (C_mn times
// 2^(sa_m + sb_n)), or both null
hipError_t launch_gemm_f64(const uint16_t *Ap, const uint16_t *Bp, double *C, int64_t M,
                           int64_t N, int64_t KB, int64_t RpadA, int64_t RpadB, int64_t ldc,
                           const int *sa, const int *sb, double alpha, double beta, int d,
                           hipStream_t s);
}  // namespace emu
