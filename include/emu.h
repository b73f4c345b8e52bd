/*
 * emu.h -- C ABI of the MI355X (gfx950) library for FP32 and FP64 GEMM
 * emulated through BF16 component products (arxiv 2609.04663).
 *
 * Problem (Sec. 3.2, Eq. gemm): C = A B with A (M x K), B (K x N), C (M x N),
 * all row-major with leading dimensions lda, ldb, ldc counted in elements.
 * emu_sgemm / emu_dgemm have no alpha/beta and no transpose: C is fully
 * overwritten.  The BLAS forms emu_sgemm_ex / emu_dgemm_ex (below) add
 * op(A), op(B) and C = alpha op(A) op(B) + beta C.
 *
 * Pointers.  A, B and C are device pointers (HIP global memory) owned by the
 * caller; A and B are only read.  C must not alias A or B.  Every call is
 * ordered on the library's current stream (emu_set_stream) and returns
 * without synchronising the host; results are ready when that stream is.
 *
 * Workspace.  The library keeps one device workspace per process (packed BF16
 * component planes, per-level exponents, a status word).  It is grown with
 * hipMalloc when a call needs more than it holds -- never on a call whose
 * sizes fit -- and freed by emu_release_workspace.  The environment variable
 * EMU_WORKSPACE_LIMIT (bytes) caps its size; a call that would exceed the cap
 * returns EMU_ENOMEM.
 *
 * Return codes.  EMU_OK on success.  EMU_EINVAL for a bad argument (checked
 * before any HIP call, nothing is launched): M, N or K negative; lda < K,
 * ldb < N, ldc < N (each at least 1); a NULL pointer for an operand with a
 * nonzero extent; nprod not one of the N_p(d) listed at emu_dgemm.  EMU_EHIP
 * when a HIP runtime call or kernel launch fails (message in emu_last_error).
 * EMU_ENOMEM when the workspace cannot be allocated.
 *
 * Degenerate sizes.  M == 0 or N == 0: nothing is done.  K == 0: C = 0.
 *
 * Input domain.  FP32 inputs: any finite value; the three-component split is
 * exact for 2^-103 <= |a| < (2 - 2^-8) 2^127 (Sec. 4.2).  FP64 inputs: the
 * BF16-range domain of Eq. (bf16rangefp64) -- 0 or 2^-126 <= |x| <=
 * (2 - 2^-7) 2^127 -- with every extracted slice a normal BF16 value
 * (Sec. 3.1, 4.3).  As in the paper there is no fallback: out-of-domain input
 * is computed anyway and reported through emu_domain_status; the call itself
 * does not fail.
 *
 * Not thread-safe: one host thread at a time may call into the library.
 */
#ifndef EMU_H
#define EMU_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EMU_OK 0
#define EMU_EINVAL 1
#define EMU_EHIP 2
#define EMU_ENOMEM 3

/* Status bits reported by emu_domain_status. */
#define EMU_STATUS_NAN 1u       /* NaN or infinity in an operand */
#define EMU_STATUS_RANGE 2u     /* finite FP64 input outside Eq. (bf16rangefp64) */
#define EMU_STATUS_SUBNORMAL 4u /* a nonzero component is subnormal in BF16 or
                                   underflowed (the split is not exact) */
#define EMU_STATUS_OVERFLOW 8u  /* a component overflowed BF16 */
#define EMU_STATUS_INEXACT 16u  /* (emu_dgemm) a retained panel product may leave
                                   FP32's exact range: for some (i, j) of the
                                   product set, 2^(vA_i + vB_j - 16) (the unit of
                                   the panel sum) is below 2^-126 or
                                   2^(vA_i + vB_j + 8) (its bound) above 2^127,
                                   so that product may be rounded or overflow in
                                   FP32 and the result is not Eq.
                                   (fp64reconstruction) with exact panel products */

#define EMU_STATUS_FALLBACK 32u /* (emu_dgemm with EMU_FALLBACK_FP64) the call's
                                   split raised a bit above and C was computed by
                                   the native FP64 fallback instead */

/* FP64 split projection constant (Eq. fp64split).  SYM (default) uses
   Sigma = 0.75 * 2^(v+45): granularity 2^(v-8) for both signs, which is the
   reading that reproduces the paper's accuracy table.  LITERAL uses
   Sigma = 2^(v+45) exactly as printed. */
#define EMU_SPLIT_SYM 0
#define EMU_SPLIT_LITERAL 1

/* Exponent scope of the FP64 split (emu_set_split_scope).
   OPERAND (default): the paper's split, one exponent chain v^(r) per operand
   (Eq. fp64split, maxima over the whole operand).
   ROWCOL: the scale-aware form the paper names as its key future step
   (Sec. 9), with stored power-of-two weights as in Eq. (ozakiscaled) at row /
   column granularity: every row m of A is divided by 2^sA_m and every column
   n of B by 2^sB_n, s = ceil(log2 max|x|) over that row or column (0 if it has
   no nonzero finite entry); the scaled operands get the operand-wide split;
   the GEMM multiplies the weights back, C_mn = 2^(sA_m + sB_n) C'_mn.  The
   scalings are exact (powers of two), so the domain becomes: finite inputs
   whose nonzero entries lie within 2^-126 of their row's (A) or column's (B)
   largest magnitude, and results that neither overflow nor underflow FP64. */
#define EMU_SCOPE_OPERAND 0
#define EMU_SCOPE_ROWCOL 1
/* KBIN: the scale-aware form extended along the reduction, for products whose
   terms differ in magnitude along k (for example some rows of B far larger
   than the others), which row and column weights cannot normalise.  With the
   ROWCOL weights sA, sB, the class of reduction index k is
     min(7, floor(-(ceil(log2 max_m |A_mk 2^-sA_m|) + ceil(log2 max_n |B_kn 2^-sB_n|)) / 8))
   (op(A), op(B); an index whose column of op(A) or row of op(B) is zero adds
   exact zeros and is left out).  The indices of each class form a group; each
   group is an emulated DGEMM of its columns of op(A) and rows of op(B) in the
   ROWCOL scope (its own weights and exponent chains), and the groups are added
   in FP64 in ascending class order, S = P_0, then S = fl(P_c + S); the
   call returns fl(fl(alpha S) + fl(beta C)).  The call synchronises its stream
   once (to size the groups) and uses workspace for the gathered groups
   (8 (M + N) K bytes) and, unless alpha = 1 and beta = 0, for S (8 M N).
   Not available to emu_dgemm_noalloc (EMU_EINVAL).  emu_split_f64 and the
   status checks behave as in ROWCOL. */
#define EMU_SCOPE_KBIN 2

/* Emulated SGEMM, Algorithm fp32 (Sec. 4.2, Eq. fp32split and fp32six):
   each FP32 operand is split into three BF16 components; the six products
   A_iB_j with i + j < 3 are evaluated with FP32 accumulation on bf16 MFMA.
   The leading product A0B0 is accumulated per reduction panel of 256 and each
   panel sum is added into an FP32 total; the five smaller products share a
   second FP32 accumulator over the whole reduction (or over each part of a
   split reduction), added to the total at the end.  A: M x K (lda), B: K x N
   (ldb), C: M x N (ldc), device pointers, FP32. */
int emu_sgemm(int64_t M, int64_t N, int64_t K, const float *A, int64_t lda, const float *B,
              int64_t ldb, float *C, int64_t ldc);

/* Emulated DGEMM, Algorithm fp64 (Sec. 4.3, Eq. fp64split, fp64productcounts,
   fp64reconstruction): each FP64 operand gets the fixed six-slice Ozaki split
   with operand-wide exponents; the nprod products A_i B_j with i, j < 6 and
   i + j < d (Eq. product-selection) are each formed in FP32 per reduction
   panel of 256 (exactly, see below), widened and added in FP64 in the order:
   panel ascending, diagonal i + j ascending, i ascending.  nprod = N_p(d):
   6, 10, 15, 21 for the paper's d = 3, 4, 5, 6 (Eq. fp64productcounts), and
   the rest of the selection sequence, 1, 3 (d = 1, 2) and 26, 30, 33, 35, 36
   (d = 7 .. 11; 36 keeps all six-by-six products, Sec. 4.3).
   A: M x K (lda), B: K x N (ldb), C: M x N (ldc), device pointers, FP64.
   For in-domain inputs every panel product is an exact FP32 value, so the
   result is independent of the order of the bf16 MFMA accumulation inside a
   panel. */
int emu_dgemm(int64_t M, int64_t N, int64_t K, const double *A, int64_t lda, const double *B,
              int64_t ldb, double *C, int64_t ldc, int nprod);

/* emu_dgemm for callers that cannot allocate device memory: code under HIP
   graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
   arguments, result and status reporting as emu_dgemm (current stream,
   current split mode and scope), but it never allocates: instead of the
   growing workspace it uses a fixed 64 MiB device array that the library
   holds on every GPU it runs on until the process ends (its address is looked
   up on the first call on each device, which also clears its status word with
   a kernel).  A call whose packed planes (2 min(d, 6) bytes per element of
   both operands, rows padded to whole tiles and K to whole k-blocks) plus a
   2 KB header and, in the ROWCOL scope, 12 bytes per row of A and column of B
   exceed 64 MiB returns EMU_ENOMEM before launching anything (square
   problems up to about M = N = K = 1500 at nprod = 21, 2100 at nprod = 6).  All calls on one GPU
   share that array: calls that overlap in time on one GPU (two streams, two
   host threads) race and must be ordered by the caller.  C, A and B are the
   caller's, as for emu_dgemm. */
int emu_dgemm_noalloc(int64_t M, int64_t N, int64_t K, const double *A, int64_t lda,
                      const double *B, int64_t ldb, double *C, int64_t ldc, int nprod);

/* BLAS forms (the "more complete BLAS semantics" of Sec. 9):
     C = alpha op(A) op(B) + beta C,  row-major, op(X) = X or X^T.
   transa, transb: 'N' (op(X) = X) or 'T' ('C' is accepted as 'T'; lower case
   too).  op(A) is M x K: A is M x K with lda >= max(1, K) for 'N', K x M with
   lda >= max(1, M) for 'T'.  op(B) is K x N: B is K x N with ldb >= max(1, N)
   for 'N', N x K with ldb >= max(1, K) for 'T'.  With P the emulated product
   (the value emu_sgemm / emu_dgemm give for op(A) op(B)), each entry becomes
   fl(alpha P) if beta == 0 -- C is then not read and may hold anything -- and
   fl(fl(alpha P) + fl(beta C)) otherwise (no fused multiply-add), so
   alpha = 1, beta = 0 is emu_sgemm / emu_dgemm exactly.  alpha == 0 or K == 0:
   A and B are not read and C = beta C (0 when beta == 0).  Transposed operands
   are packed from their stored layout directly, so op(A) op(B) gives the same
   bits as the plain call on explicitly transposed copies.  Errors as for
   emu_sgemm / emu_dgemm, plus EMU_EINVAL for another transa / transb. */
int emu_sgemm_ex(char transa, char transb, int64_t M, int64_t N, int64_t K, float alpha,
                 const float *A, int64_t lda, const float *B, int64_t ldb, float beta, float *C,
                 int64_t ldc);
int emu_dgemm_ex(char transa, char transb, int64_t M, int64_t N, int64_t K, double alpha,
                 const double *A, int64_t lda, const double *B, int64_t ldb, double beta,
                 double *C, int64_t ldc, int nprod);

/* Fallback of the emulated DGEMM for inputs its split cannot represent (the
   "fallback handling" of Sec. 9 and the "fallback extension" of Sec. 4.3),
   for subsequent emu_dgemm, emu_dgemm_ex and emu_dgemm_noalloc calls.
   EMU_FALLBACK_NONE (default): as in the paper, out-of-domain input is
   computed anyway and only reported.  EMU_FALLBACK_FP64: when the split of
   the call raises any EMU_STATUS_* bit (NaN or infinity, an entry outside
   Eq. (bf16rangefp64) in the current scope, a subnormal, underflowed or
   overflowed slice, a panel product that may be inexact in FP32), C is
   recomputed as alpha op(A) op(B) + beta C by a plain FP64 GEMM (fused
   multiply-adds, its own summation order) and EMU_STATUS_FALLBACK is reported
   as well.  The decision is taken on the device: no host synchronisation; the
   armed mode costs a kernel launch per call that does nothing unless the
   fallback is needed, plus, for beta != 0, a copy of C in the workspace.
   EMU_EINVAL for any other value. */
#define EMU_FALLBACK_NONE 0
#define EMU_FALLBACK_FP64 1
int emu_set_fallback(int mode);

/* How subsequent emu_sgemm and emu_sgemm_ex calls split their operands
   (Eq. fp32split; Sec. 6.2 weighs the two ways):
   EMU_SGEMM_SPLIT_PASS (default): a split kernel writes the three BF16 planes
   of both operands to the workspace, and the product kernel reads them;
   EMU_SGEMM_SPLIT_STREAMED: the product kernel reads op(A) and op(B) in FP32
   and splits every k-block itself, in each workgroup that uses it, with the
   split kernel's arithmetic (128 x 128 output tiles): no planes in HBM,
   workspace only for split-reduction partial sums, the same status bits, and
   the same result bits whenever both ways cut the reduction into the same
   number of parts.  EMU_EINVAL for any other value. */
#define EMU_SGEMM_SPLIT_PASS 0
#define EMU_SGEMM_SPLIT_STREAMED 1
int emu_set_sgemm_split(int mode);

/* Stream for subsequent calls (a hipStream_t); NULL selects the default
   stream.  Switching streams orders the new stream after the work already
   queued on the previous one (an event dependency, no host synchronisation),
   since every call uses the one workspace.  EMU_OK, or EMU_EHIP if the event
   calls fail. */
int emu_set_stream(void *hip_stream);

/* Projection constant of the FP64 split for subsequent emu_dgemm and
   emu_split_f64 calls: EMU_SPLIT_SYM (default) or EMU_SPLIT_LITERAL.
   EMU_EINVAL for any other value. */
int emu_set_split_mode(int mode);

/* Exponent scope of the FP64 split for subsequent emu_dgemm and emu_split_f64
   calls: EMU_SCOPE_OPERAND (default), EMU_SCOPE_ROWCOL or EMU_SCOPE_KBIN (see above).  In the
   ROWCOL scope the domain checks behind EMU_STATUS_RANGE apply to the scaled
   operands.  EMU_EINVAL for any other value. */
int emu_set_split_scope(int scope);

/* Synchronises the current stream, stores in *flags the EMU_STATUS_* bits
   accumulated by all calls since the previous emu_domain_status, and clears
   them.  EMU_EINVAL if flags is NULL. */
int emu_domain_status(unsigned *flags);

/* Message of the last failing call (empty string if none).  Owned by the
   library, valid until the next call. */
const char *emu_last_error(void);

/* Frees the workspace (synchronises the device first).  The next call
   allocates again. */
int emu_release_workspace(void);

/* Bytes currently held by the workspace (0 after emu_release_workspace). */
int64_t emu_workspace_bytes(void);

/* Test hook: the FP32 split of Eq. (fp32split) as the GEMM consumes it.
   X is an R x Cc row-major FP32 device matrix (ldx).  as_b = 0 runs the
   A-operand pack (rows of X are GEMM rows), as_b = 1 the B-operand pack (X is
   K x N and is packed transposed).  comps (device, uint16 BF16 bit patterns)
   receives [3][R][Cc], plane-major, in X's own orientation, unpacked from the
   packed buffer.  Errors as above. */
int emu_split_f32(int64_t R, int64_t Cc, const float *X, int64_t ldx, int as_b, uint16_t *comps);

/* Test hook: the FP64 split of Eq. (fp64split) as the GEMM consumes it.
   X is R x Cc row-major FP64 (device, ldx); as_b as for emu_split_f32.
   slices (device) receives [6][R][Cc] BF16 bit patterns; v (device, int32[6])
   receives v^(r) = ceil(log2 max|X^(r)|) per level, INT32_MIN for a level
   whose residual is identically zero.  In the ROWCOL scope these are the
   slices and exponents of the scaled operand (rows of X scaled when as_b = 0,
   columns when as_b = 1). */
int emu_split_f64(int64_t R, int64_t Cc, const double *X, int64_t ldx, int as_b,
                  uint16_t *slices, int32_t *v);

/* Test hook: the weights of the ROWCOL scope.  X is R x Cc row-major FP64
   (device, ldx); s (device, int32) receives ceil(log2 max|x|) over each row
   (by_col = 0, R entries) or each column (by_col = 1, Cc entries), ignoring
   non-finite entries, 0 for a row or column without a nonzero finite entry.
   EMU_EINVAL for negative sizes, ldx < max(1, Cc), by_col not 0 or 1, or a
   NULL pointer with nonzero extent. */
int emu_scale_exponents(int64_t R, int64_t Cc, const double *X, int64_t ldx, int by_col,
                        int32_t *s);

/* Phase timing, the analog of the paper's runtime breakdown (Sec. 8.4):
   decomposition + packing versus the component-product GEMM with its
   reconstruction.  emu_profile_enable(1) creates a pool of HIP events for
   4096 calls (the only allocation, done here, outside any timed region); from
   then on every emu_sgemm / emu_dgemm records three events on its stream:
   before its split kernels, between them and its GEMM kernel, and after the
   GEMM kernel.  emu_profile_read synchronises the device, writes the split/pack
   and GEMM milliseconds of the profiled calls since the previous read, oldest
   first, into split_ms[i] and gemm_ms[i] for i < min(cap, *calls) (host arrays
   owned by the caller), stores the number of such calls in *calls and starts
   over.  Calls made while the pool is full are not profiled.
   emu_profile_enable(0) destroys the pool.  EMU_EINVAL if calls is NULL, or if
   cap > 0 and an array is NULL. */
int emu_profile_enable(int on);
int emu_profile_read(int64_t cap, double *split_ms, double *gemm_ms, int64_t *calls);

#ifdef __cplusplus
}
#endif

#endif /* EMU_H */
