/*
 * CPU oracle for FP32 / FP64 GEMM emulated through BF16 component products
 * (arxiv 2609.04663).  TEST INFRASTRUCTURE ONLY: only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load this library.  It shares
 * no code with the HIP implementation and is deliberately plain and slow.
 *
 * Everything here follows the paper step by step, in the paper's notation:
 *   - BF16 rounding fl_BF16: round to nearest, ties to even (Sec. 3.1, 4.1).
 *   - Split_FP32: three-component residual split, Eq. (fp32split), Sec. 4.2.
 *   - Split_FP64: fixed six-slice simplified Ozaki split, Eq. (fp64split),
 *     Sec. 4.3, with the operand-wide maximum of Eq. (fp64split).
 *   - FP32 reconstruction: the six products of Eq. (fp32six) accumulated in
 *     FP32 in the operand-reuse order of Eq. (fp32reuseorder), per reduction
 *     panel of length kc (B_K = 256), panel results added into an FP32 block
 *     accumulator (Sec. 6.2 and 6.3).
 *   - FP64 reconstruction: Eq. (fp64reconstruction) / Algorithm fp64, each
 *     FP32 component-product panel result widened and added in FP64, panel by
 *     panel (Sec. 6.3), diagonals in increasing order, i increasing inside a
 *     diagonal.
 *   - References: a plain FP64 GEMM and a double-double dot product (Dot2 of
 *     Ogita, Rump and Oishi 2005: TwoProduct via fma, TwoSum accumulation).
 *
 * Projection constant of the FP64 split.  With Sigma = 2^(v+rho), rho = 45, the
 * add-subtract projection keeps granularity 2^(v-7) for non-negative residuals
 * and 2^(v-8) for negative ones.  That literal form does not reproduce the
 * paper's own accuracy table; Sigma = 0.75 * 2^(v+45) keeps x + Sigma in one
 * binade and gives granularity 2^(v-8) for both signs, which does.  Mode
 * ORC_SPLIT_SYM (0, default) uses 0.75 * 2^(v+45); ORC_SPLIT_LITERAL (1) uses
 * 2^(v+45).  Only the constant differs.
 *
 * Status bits returned by the split and GEMM routines:
 *   1  NaN or infinity in an operand
 *   2  finite FP64 input outside the BF16-range domain, Eq. (bf16rangefp64)
 *   4  a nonzero component is subnormal in BF16 (or rounded away to zero)
 *   8  a component overflowed BF16
 *  16  (FP64 path) a panel component-product sum is not exactly an FP32 value
 */
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_NAN 1u
#define ORC_RANGE 2u
#define ORC_SUBNORMAL 4u
#define ORC_OVERFLOW 8u
#define ORC_INEXACT32 16u

#define ORC_SPLIT_SYM 0
#define ORC_SPLIT_LITERAL 1

typedef int64_t i64;

static float f32_of_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_of_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* Exact value of a BF16 bit pattern.  BF16 is the upper half of binary32. */
float orc_bf16_value(uint16_t h) { return f32_of_bits((uint32_t)h << 16); }

/* Value used for distance comparisons: the pattern one step past the largest
   finite BF16 (exponent field all ones, zero fraction) stands for 2^128. */
static double bf16_dist_value(uint32_t pattern32) {
    if ((pattern32 & 0x7FFFFFFFu) == 0x7F800000u)
        return (pattern32 >> 31) ? -ldexp(1.0, 128) : ldexp(1.0, 128);
    return (double)f32_of_bits(pattern32);
}

/* fl_BF16 of a binary32 value: the nearer of the two BF16 values that bracket
   a (BF16 values are the binary32 values whose low 16 bits are zero), ties to
   the one whose last retained fraction bit is zero.  Overflow gives infinity. */
uint16_t orc_bf16_rne_f32(float a) {
    uint32_t u = bits_of_f32(a);
    if (isnan(a)) return (uint16_t)((u >> 16) | 0x0040u);
    if (isinf(a)) return (uint16_t)(u >> 16);
    uint32_t lo = u & 0xFFFF0000u;          /* toward zero */
    if (lo == u) return (uint16_t)(u >> 16);
    uint32_t hi = lo + 0x10000u;            /* next BF16 away from zero */
    double dlo = fabs((double)a - bf16_dist_value(lo));
    double dhi = fabs(bf16_dist_value(hi) - (double)a);
    if (dlo < dhi) return (uint16_t)(lo >> 16);
    if (dhi < dlo) return (uint16_t)(hi >> 16);
    return ((lo >> 16) & 1u) ? (uint16_t)(hi >> 16) : (uint16_t)(lo >> 16);
}

/* fl_BF16 of a binary64 value with a single rounding (no detour through
   binary32): the BF16 spacing at |z| is 2^(floor(log2|z|) - 7), and never less
   than the subnormal spacing 2^-133. */
uint16_t orc_bf16_rne_f64(double z) {
    if (isnan(z)) return 0x7FC0u;
    uint16_t sign = signbit(z) ? 0x8000u : 0u;
    if (isinf(z)) return (uint16_t)(sign | 0x7F80u);
    if (z == 0.0) return sign;
    double az = fabs(z);
    int e;
    (void)frexp(az, &e);                    /* az in [2^(e-1), 2^e) */
    int q = e - 1;
    if (q < -126) q = -126;
    double spacing = ldexp(1.0, q - 7);
    double r = nearbyint(az / spacing) * spacing;   /* default mode: ties to even */
    if (r > ldexp(255.0, 120)) return (uint16_t)(sign | 0x7F80u);   /* beyond the largest BF16 */
    float rf = (float)r;                    /* exact: r is a BF16 value */
    return (uint16_t)(sign | (bits_of_f32(rf) >> 16));
}

static unsigned classify_bf16(uint16_t h, int source_nonzero) {
    unsigned st = 0;
    uint16_t ex = (uint16_t)((h >> 7) & 0xFF), fr = (uint16_t)(h & 0x7F);
    if (ex == 0xFF) st |= ORC_OVERFLOW;
    else if (ex == 0 && fr != 0) st |= ORC_SUBNORMAL;
    else if (ex == 0 && fr == 0 && source_nonzero) st |= ORC_SUBNORMAL;
    return st;
}

/* Threads of the OpenMP loops below (the benchmark's one-core baseline). */
void orc_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------- */
/* Split_FP32, Eq. (fp32split): A_r = fl_BF16(A^(r)), A^(r+1) = fl_32(A^(r) - A_r),
   r = 0, 1, 2.  comps is [3][R][C] (plane-major, row-major planes). */
unsigned orc_split_f32(i64 R, i64 C, const float *X, i64 ldx, uint16_t *comps) {
    unsigned status = 0;
    const i64 plane = R * C;
#pragma omp parallel for reduction(| : status) schedule(static)
    for (i64 r = 0; r < R; ++r) {
        for (i64 c = 0; c < C; ++c) {
            float a = X[r * ldx + c];
            if (!isfinite(a)) status |= ORC_NAN;
            float res = a;
            for (int t = 0; t < 3; ++t) {
                uint16_t h = orc_bf16_rne_f32(res);
                comps[t * plane + r * C + c] = h;
                if (isfinite(a)) status |= classify_bf16(h, res != 0.0f);
                res = res - orc_bf16_value(h);
            }
            /* outside 2^-103 <= |a| < (2 - 2^-8) 2^127 the three components may
               not represent a exactly; report that as an underflowed component */
            if (isfinite(a) && isfinite(res) && res != 0.0f) status |= ORC_SUBNORMAL;
        }
    }
    return status;
}

/* v = ceil(log2 m) for m > 0, exactly: m = f 2^e with f in [1/2, 1). */
static int ceil_log2(double m) {
    int e;
    double f = frexp(m, &e);
    return (f == 0.5) ? e - 1 : e;
}

static int in_bf16_range_f64(double x) {
    if (x == 0.0) return 1;
    double ax = fabs(x);
    return ax >= ldexp(1.0, -126) && ax <= ldexp(255.0, 120);
}

/* Split_FP64, Eq. (fp64split), six slices, operand-wide maximum.
   slices is [6][R][C] BF16 bit patterns; v[6] receives v_A^(r) (INT_MIN for a
   level whose residual is entirely zero); resid (optional, [R][C]) receives the
   terminal residual A^(6). */
unsigned orc_split_f64(i64 R, i64 C, const double *X, i64 ldx, int mode,
                       uint16_t *slices, int32_t *v, double *resid) {
    unsigned status = 0;
    const i64 plane = R * C;
    double *W = (double *)malloc((size_t)(plane > 0 ? plane : 1) * sizeof(double));
    if (!W) return 0xFFFFFFFFu;
#pragma omp parallel for reduction(| : status) schedule(static)
    for (i64 r = 0; r < R; ++r)
        for (i64 c = 0; c < C; ++c) {
            double x = X[r * ldx + c];
            if (!isfinite(x)) status |= ORC_NAN;
            else if (!in_bf16_range_f64(x)) status |= ORC_RANGE;
            W[r * C + c] = x;
        }
    int zero_from = 6;
    for (int lev = 0; lev < 6; ++lev) {
        double m = 0.0;
#pragma omp parallel for reduction(max : m) schedule(static)
        for (i64 i = 0; i < plane; ++i) {
            double a = fabs(W[i]);
            if (a > m) m = a;           /* NaN compares false and is skipped */
        }
        if (m == 0.0 || !isfinite(m)) { zero_from = lev; break; }
        int vr = ceil_log2(m);
        v[lev] = vr;
        double sigma = (mode == ORC_SPLIT_LITERAL) ? ldexp(1.0, vr + 45) : ldexp(0.75, vr + 45);
        unsigned st = 0;
#pragma omp parallel for reduction(| : st) schedule(static)
        for (i64 i = 0; i < plane; ++i) {
            double a = W[i];
            volatile double t = a + sigma;  /* fl_64(A^(r) + Sigma) */
            double z = t - sigma;           /* Z = fl_64(t - Sigma) */
            uint16_t h = orc_bf16_rne_f64(z);   /* A_r = fl_BF16(Z) */
            slices[lev * plane + i] = h;
            st |= classify_bf16(h, z != 0.0);
            W[i] = a - (double)orc_bf16_value(h);   /* A^(r+1) = fl_64(A^(r) - A_r) */
        }
        status |= st;
    }
    for (int lev = zero_from; lev < 6; ++lev) {
        v[lev] = INT32_MIN;
        memset(slices + (size_t)lev * plane, 0, (size_t)plane * sizeof(uint16_t));
    }
    if (resid) memcpy(resid, W, (size_t)plane * sizeof(double));
    free(W);
    return status;
}

/* ------------------------------------------------------------------------- */
/* Exact accumulation of BF16 x BF16 products and one correct rounding.

   fl_32(A_i B_j) over a reduction panel is the FP32 value nearest to the exact
   panel dot product (ties to even).  The exact sum is held in a fixed-point
   two's-complement integer of XL_LIMBS 64-bit limbs whose least significant bit
   weighs 2^XL_LSB.  Every product of two finite BF16 values (subnormals
   included) is an integer of at most 16 bits times 2^e with e >= 2*(-133), and
   is below 2^256, so the window [2^-266, 2^446) with 64 guard bits of carry
   room holds any panel of up to 2^60 terms exactly. */
#define XL_LIMBS 12
#define XL_LSB (-266)

typedef struct { uint64_t w[XL_LIMBS]; } xacc;

static void xacc_zero(xacc *a) { memset(a, 0, sizeof(*a)); }

/* a += s * 2^e, s a signed integer with |s| < 2^17, e >= XL_LSB. */
static void xacc_add(xacc *a, int64_t s, int e) {
    if (s == 0) return;
    int sh = e - XL_LSB;
    int limb = sh / 64, off = sh % 64;
    uint64_t mag = (uint64_t)(s < 0 ? -s : s);
    uint64_t lo = mag << off;
    uint64_t hi = off ? (mag >> (64 - off)) : 0;
    if (s > 0) {
        uint64_t c = 0;
        for (int t = limb; t < XL_LIMBS; ++t) {
            uint64_t add = (t == limb) ? lo : (t == limb + 1) ? hi : 0;
            uint64_t x = a->w[t] + add;
            uint64_t c1 = x < add;
            uint64_t y = x + c;
            uint64_t c2 = y < c;
            a->w[t] = y;
            c = c1 | c2;
            if (t > limb + 1 && c == 0) break;
        }
    } else {
        uint64_t b = 0;
        for (int t = limb; t < XL_LIMBS; ++t) {
            uint64_t sub = (t == limb) ? lo : (t == limb + 1) ? hi : 0;
            uint64_t x = a->w[t] - sub;
            uint64_t b1 = a->w[t] < sub;
            uint64_t y = x - b;
            uint64_t b2 = x < b;
            a->w[t] = y;
            b = b1 | b2;
            if (t > limb + 1 && b == 0) break;
        }
    }
}

/* Split a finite BF16 value into integer significand and exponent: v = s 2^e. */
static void bf16_parts(uint16_t h, int64_t *s, int *e) {
    int ex = (h >> 7) & 0xFF, fr = h & 0x7F, neg = h >> 15;
    int64_t m;
    if (ex == 0) { m = fr; *e = -126 - 7; }
    else { m = 128 | fr; *e = ex - 127 - 7; }
    *s = neg ? -m : m;
}

static void xacc_add_product(xacc *a, uint16_t x, uint16_t y) {
    int64_t sx, sy;
    int ex, ey;
    bf16_parts(x, &sx, &ex);
    bf16_parts(y, &sy, &ey);
    xacc_add(a, sx * sy, ex + ey);
}

/* Nearest binary32 to the exact value held in a (ties to even). */
static float xacc_round_f32(const xacc *a) {
    xacc m = *a;
    int neg = (int)(m.w[XL_LIMBS - 1] >> 63);
    if (neg) {                                   /* magnitude = two's complement */
        uint64_t c = 1;
        for (int t = 0; t < XL_LIMBS; ++t) {
            uint64_t x = ~m.w[t] + c;
            c = (c && x == 0);
            m.w[t] = x;
        }
    }
    int top = -1;
    for (int t = XL_LIMBS - 1; t >= 0 && top < 0; --t)
        if (m.w[t]) top = t * 64 + 63 - __builtin_clzll(m.w[t]);
    if (top < 0) return neg ? -0.0f : 0.0f;
    int e_top = top + XL_LSB;                    /* value in [2^e_top, 2^(e_top+1)) */
    int q = e_top - 23;                          /* binary32 spacing at this magnitude */
    if (q < -149) q = -149;                      /* subnormal spacing */
    int cut = q - XL_LSB;                        /* bit index of the last kept bit */
    uint64_t kept = 0;                           /* bits [cut, top] (at most 24 bits) */
    for (int b = top; b >= cut; --b) {
        int bit = (b >= 0) ? (int)((m.w[b / 64] >> (b % 64)) & 1u) : 0;
        kept = (kept << 1) | (uint64_t)bit;
    }
    int guard = 0, sticky = 0;
    if (cut - 1 >= 0) guard = (int)((m.w[(cut - 1) / 64] >> ((cut - 1) % 64)) & 1u);
    for (int b = cut - 2; b >= 0 && !sticky; --b)
        if ((m.w[b / 64] >> (b % 64)) & 1u) sticky = 1;
    if (guard && (sticky || (kept & 1u))) kept += 1;
    double r = ldexp((double)kept, q);           /* exact: kept <= 2^24 */
    float f = (float)r;                          /* exact, or overflow to infinity */
    return neg ? -f : f;
}

/* Whether the exact value held in a equals the finite binary32 value f. */
static int xacc_is_f32(const xacc *a, float f) {
    if (!isfinite(f)) return 0;
    xacc d = *a;
    uint32_t u = bits_of_f32(f);
    int neg = (int)(u >> 31), ex = (int)((u >> 23) & 0xFF);
    int64_t mant = (int64_t)(u & 0x7FFFFFu);
    int e;
    if (ex == 0) e = -149; else { mant |= 0x800000; e = ex - 150; }
    /* subtract f in at most two pieces of < 2^17 each */
    int64_t hi = mant >> 12, lo = mant & 0xFFF;
    if (neg) { hi = -hi; lo = -lo; }
    xacc_add(&d, -hi, e + 12);
    xacc_add(&d, -lo, e);
    for (int t = 0; t < XL_LIMBS; ++t) if (d.w[t]) return 0;
    return 1;
}

/* Emulated SGEMM, Algorithm fp32, evaluated as Sec. 6.2/6.3 execute it: per
   reduction panel of length kc, the six retained component products of
   Eq. (fp32six) are each retained in FP32 (fl_32 of the panel dot product) and
   summed in FP32 in the operand-reuse order of Eq. (fp32reuseorder); each panel
   result is added in FP32 to the block accumulator. */

/* Operand-reuse order of Eq. (fp32reuseorder): A1B1, A1B0, A2B0, A0B0, A0B1, A0B2. */
static const int FP32_ORDER[6][2] = {{1, 1}, {1, 0}, {2, 0}, {0, 0}, {0, 1}, {0, 2}};

/* Components as BF16 bit patterns: Av[t][m][k], Bv[t][k][n]. */
static float sgemm_entry(i64 K, i64 kc, const uint16_t *Av, const uint16_t *Bv, i64 M, i64 N,
                         i64 m, i64 n) {
    float blk = 0.0f;                               /* FP32 block accumulator */
    for (i64 p0 = 0; p0 < K; p0 += kc) {
        i64 p1 = p0 + kc < K ? p0 + kc : K;
        float t = 0.0f;                             /* panel result in FP32 */
        for (int q = 0; q < 6; ++q) {
            const uint16_t *Ai = Av + (size_t)FP32_ORDER[q][0] * M * K + (size_t)m * K;
            const uint16_t *Bj = Bv + (size_t)FP32_ORDER[q][1] * K * N + n;
            xacc x;
            xacc_zero(&x);
            for (i64 k = p0; k < p1; ++k) xacc_add_product(&x, Ai[k], Bj[(size_t)k * N]);
            t = t + xacc_round_f32(&x);             /* fl_32(A_i B_j), summed in FP32 */
        }
        blk = blk + t;
    }
    return blk;
}

static unsigned sgemm_prepare(i64 M, i64 N, i64 K, const float *A, i64 lda, const float *B,
                              i64 ldb, uint16_t **Av, uint16_t **Bv) {
    *Av = (uint16_t *)malloc((size_t)(3 * M * K + 1) * 2);
    *Bv = (uint16_t *)malloc((size_t)(3 * K * N + 1) * 2);
    return orc_split_f32(M, K, A, lda, *Av) | orc_split_f32(K, N, B, ldb, *Bv);
}

unsigned orc_emu_sgemm(i64 M, i64 N, i64 K, const float *A, i64 lda, const float *B, i64 ldb,
                       float *C, i64 ldc, i64 kc) {
    uint16_t *Av, *Bv;
    unsigned st = sgemm_prepare(M, N, K, A, lda, B, ldb, &Av, &Bv);
#pragma omp parallel for schedule(dynamic, 1)
    for (i64 m = 0; m < M; ++m)
        for (i64 n = 0; n < N; ++n) C[m * ldc + n] = sgemm_entry(K, kc, Av, Bv, M, N, m, n);
    free(Av);
    free(Bv);
    return st;
}

/* Selected entries (rows[e], cols[e]) of the emulated SGEMM; the splits still
   cover the whole operands. */
unsigned orc_emu_sgemm_entries(i64 M, i64 N, i64 K, const float *A, i64 lda, const float *B,
                               i64 ldb, i64 nent, const i64 *rows, const i64 *cols, float *out,
                               i64 kc) {
    uint16_t *Av, *Bv;
    unsigned st = sgemm_prepare(M, N, K, A, lda, B, ldb, &Av, &Bv);
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 e = 0; e < nent; ++e) out[e] = sgemm_entry(K, kc, Av, Bv, M, N, rows[e], cols[e]);
    free(Av);
    free(Bv);
    return st;
}

/* Selected entries from components already split by orc_split_f32:
   Av [3][M][K], Bv [3][K][N] (the benchmark times the split and the entries
   apart). */
void orc_sgemm_entries_from_comps(i64 M, i64 N, i64 K, const uint16_t *Av, const uint16_t *Bv,
                                  i64 nent, const i64 *rows, const i64 *cols, float *out, i64 kc) {
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 e = 0; e < nent; ++e) out[e] = sgemm_entry(K, kc, Av, Bv, M, N, rows[e], cols[e]);
}

/* ------------------------------------------------------------------------- */
/* Emulated DGEMM, Algorithm fp64 / Eq. (fp64reconstruction). */

/* N_p(d) = |S_d| of Eq. (product-selection) with six slices per operand,
   S_d = {(i, j) : 0 <= i, j < 6, i + j < d}, for d = 1 .. 11 (d = 11 keeps all
   36 products); the paper evaluates d = 3 .. 6 (Eq. fp64productcounts). */
static int nprod_to_d(int nprod) {
    for (int d = 1; d <= 11; ++d) {
        int n = 0;
        for (int i = 0; i < 6; ++i)
            for (int j = 0; j < 6; ++j)
                if (i + j < d) ++n;
        if (n == nprod) return d;
    }
    return -1;
}

static double dgemm_entry(i64 K, i64 kc, int d, const uint16_t *Av, const uint16_t *Bv, i64 M,
                          i64 N, i64 m, i64 n, unsigned *st) {
    double c = 0.0;                                 /* FP64 output accumulator */
    for (i64 p0 = 0; p0 < K; p0 += kc) {
        i64 p1 = p0 + kc < K ? p0 + kc : K;
        for (int l = 0; l < d; ++l) {               /* diagonal l = i + j */
            for (int i = 0; i <= l; ++i) {
                int j = l - i;
                if (i > 5 || j > 5) continue;       /* six slices per operand */
                const uint16_t *Ai = Av + (size_t)i * M * K + (size_t)m * K;
                const uint16_t *Bj = Bv + (size_t)j * K * N + n;
                xacc x;
                xacc_zero(&x);
                for (i64 k = p0; k < p1; ++k) xacc_add_product(&x, Ai[k], Bj[(size_t)k * N]);
                float p32 = xacc_round_f32(&x);     /* fl_32 of the panel product */
                if (!xacc_is_f32(&x, p32)) *st |= ORC_INEXACT32;
                c = c + (double)p32;                /* widen exactly, add in FP64 */
            }
        }
    }
    return c;
}

static unsigned dgemm_prepare(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B,
                              i64 ldb, int mode, uint16_t **Av, uint16_t **Bv, int32_t *vA,
                              int32_t *vB) {
    *Av = (uint16_t *)malloc((size_t)(6 * M * K + 1) * 2);
    *Bv = (uint16_t *)malloc((size_t)(6 * K * N + 1) * 2);
    unsigned st = orc_split_f64(M, K, A, lda, mode, *Av, vA, NULL);
    st |= orc_split_f64(K, N, B, ldb, mode, *Bv, vB, NULL);
    return st;
}

unsigned orc_emu_dgemm(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B,
                       i64 ldb, double *C, i64 ldc, int nprod, int mode, i64 kc) {
    int d = nprod_to_d(nprod);
    if (d < 0) return 0xFFFFFFFFu;
    uint16_t *Av, *Bv;
    int32_t vA[6], vB[6];
    unsigned st = dgemm_prepare(M, N, K, A, lda, B, ldb, mode, &Av, &Bv, vA, vB);
    unsigned st2 = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : st2)
    for (i64 m = 0; m < M; ++m) {
        unsigned s = 0;
        for (i64 n = 0; n < N; ++n) C[m * ldc + n] = dgemm_entry(K, kc, d, Av, Bv, M, N, m, n, &s);
        st2 |= s;
    }
    free(Av);
    free(Bv);
    return st | st2;
}

unsigned orc_emu_dgemm_entries(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B,
                               i64 ldb, i64 nent, const i64 *rows, const i64 *cols, double *out,
                               int nprod, int mode, i64 kc) {
    int d = nprod_to_d(nprod);
    if (d < 0) return 0xFFFFFFFFu;
    uint16_t *Av, *Bv;
    int32_t vA[6], vB[6];
    unsigned st = dgemm_prepare(M, N, K, A, lda, B, ldb, mode, &Av, &Bv, vA, vB);
    unsigned st2 = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : st2)
    for (i64 e = 0; e < nent; ++e) {
        unsigned s = 0;
        out[e] = dgemm_entry(K, kc, d, Av, Bv, M, N, rows[e], cols[e], &s);
        st2 |= s;
    }
    free(Av);
    free(Bv);
    return st | st2;
}

/* Selected entries from slices already split by orc_split_f64: Av [6][M][K],
   Bv [6][K][N]; returns the inexact-panel status (bit 16). */
unsigned orc_dgemm_entries_from_slices(i64 M, i64 N, i64 K, const uint16_t *Av,
                                       const uint16_t *Bv, i64 nent, const i64 *rows,
                                       const i64 *cols, double *out, int nprod, i64 kc) {
    int d = nprod_to_d(nprod);
    if (d < 0) return 0xFFFFFFFFu;
    unsigned st2 = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : st2)
    for (i64 e = 0; e < nent; ++e) {
        unsigned s = 0;
        out[e] = dgemm_entry(K, kc, d, Av, Bv, M, N, rows[e], cols[e], &s);
        st2 |= s;
    }
    return st2;
}

/* ------------------------------------------------------------------------- */
/* References. */

/* Plain FP64 GEMM, ascending k.  For FP32 inputs (passed widened) every product
   is exact and the only error is the FP64 summation, about K * 2^-53. */
void orc_ref_gemm_f64(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B, i64 ldb,
                      double *C, i64 ldc) {
#pragma omp parallel for schedule(dynamic, 1)
    for (i64 m = 0; m < M; ++m)
        for (i64 n = 0; n < N; ++n) {
            double s = 0.0;
            for (i64 k = 0; k < K; ++k) s += A[m * lda + k] * B[k * ldb + n];
            C[m * ldc + n] = s;
        }
}

/* Error-free transformations (Knuth TwoSum; TwoProduct through one fma). */
static void two_sum(double a, double b, double *s, double *e) {
    double x = a + b;
    double z = x - a;
    *e = (a - (x - z)) + (b - z);
    *s = x;
}

static double dot2(i64 K, const double *a, i64 sa, const double *b, i64 sb, double *lo) {
    double s = 0.0, c = 0.0;
    for (i64 k = 0; k < K; ++k) {
        double x = a[k * sa], y = b[k * sb];
        double p = x * y;
        double pe = fma(x, y, -p);
        double t, te;
        two_sum(s, p, &t, &te);
        s = t;
        c += pe + te;
    }
    double hi, l;
    two_sum(s, c, &hi, &l);
    *lo = l;
    return hi;
}

/* Double-double reference C ~ Chi + Clo, accurate as if computed in twice the
   working precision and rounded (Ogita, Rump, Oishi, Dot2). */
void orc_ref_gemm_dd(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B, i64 ldb,
                     double *Chi, double *Clo, i64 ldc) {
#pragma omp parallel for schedule(dynamic, 1)
    for (i64 m = 0; m < M; ++m)
        for (i64 n = 0; n < N; ++n) {
            double lo;
            Chi[m * ldc + n] = dot2(K, A + m * lda, 1, B + n, ldb, &lo);
            Clo[m * ldc + n] = lo;
        }
}

void orc_ref_dd_entries(i64 M, i64 N, i64 K, const double *A, i64 lda, const double *B,
                        i64 ldb, i64 nent, const i64 *rows, const i64 *cols, double *hi,
                        double *lo) {
    (void)M;
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 e = 0; e < nent; ++e) {
        double l;
        hi[e] = dot2(K, A + rows[e] * lda, 1, B + cols[e], ldb, &l);
        lo[e] = l;
    }
}

/* Entrywise |A||B| in FP64 (the denominator of the GEMM-scaled error). */
void orc_absprod_entries(i64 K, const double *A, i64 lda, const double *B, i64 ldb, i64 nent,
                         const i64 *rows, const i64 *cols, double *out) {
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 e = 0; e < nent; ++e) {
        double s = 0.0;
        for (i64 k = 0; k < K; ++k) s += fabs(A[rows[e] * lda + k]) * fabs(B[k * ldb + cols[e]]);
        out[e] = s;
    }
}

/* fl_32 of the exact dot product of two BF16 vectors (the per-panel component
   product of the FP32 and FP64 reconstructions, exposed for the pins). */
float orc_dot_bf16_f32(i64 n, const uint16_t *x, const uint16_t *y) {
    xacc a;
    xacc_zero(&a);
    for (i64 k = 0; k < n; ++k) xacc_add_product(&a, x[k], y[k]);
    return xacc_round_f32(&a);
}
