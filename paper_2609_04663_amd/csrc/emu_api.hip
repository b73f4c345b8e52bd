// Host side of the C ABI declared in include/emu.h: argument validation,
// the device workspace, launch sequencing on the current stream, status and
// error reporting.  Every entry point validates its arguments before any HIP
// call; no entry point synchronises the host except emu_domain_status and
// emu_release_workspace.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/emu.h"
#include "emu_internal.h"

namespace emu {

int device_cu_count() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n < 1)
            n = 256;
        cus = n;
    }
    return cus;
}

}  // namespace emu

// Fixed scratch of the allocation-free entry point emu_dgemm_noalloc: header
// (status word, split state), packed planes and scale-aware weights of one
// call.  A file-scope device array: every GPU the library runs on holds its
// own copy from the library's load until the process ends.  In host code the
// name `scratch` only stands in for the symbol; the device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
constexpr size_t NOALLOC_BYTES = (size_t)64 << 20;
static __device__ __align__(256) char scratch[NOALLOC_BYTES];

namespace {

using namespace emu;

hipStream_t g_stream = nullptr;
hipEvent_t g_switch_event = nullptr;   // orders a new stream after the previous one
int g_split_mode = EMU_SPLIT_SYM;
int g_split_scope = EMU_SCOPE_OPERAND;
int g_fallback = EMU_FALLBACK_NONE;
int g_sgemm_split = EMU_SGEMM_SPLIT_PASS;
std::string g_err;

// Workspace: [status word (offset 0), the FP64 split state slots of two
//            operands (offset 128): 2 KB header][operand A planes][operand B planes].
// Grown only when a call needs more; the status word is preserved across growth.
struct Workspace {
    char *base = nullptr;
    size_t bytes = 0;
} g_ws;

constexpr size_t HDR = 2048;
static_assert(128 + 2 * F64_SLOTS * sizeof(F64SplitState) <= HDR, "workspace header");

int fail(int code, const char *msg) {
    g_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return EMU_EHIP;
}

size_t workspace_limit() {
    const char *s = getenv("EMU_WORKSPACE_LIMIT");
    if (!s || !*s) return (size_t)-1;
    return (size_t)strtoull(s, nullptr, 0);
}

int ensure_workspace(size_t need) {
    need += HDR;
    if (need <= g_ws.bytes) return EMU_OK;
    if (need > workspace_limit()) return fail(EMU_ENOMEM, "workspace would exceed EMU_WORKSPACE_LIMIT");
    unsigned status = 0;
    if (g_ws.base) {
        hipError_t e = hipStreamSynchronize(g_stream);
        if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
        e = hipMemcpy(&status, g_ws.base, sizeof(status), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy(status)");
        e = hipFree(g_ws.base);
        g_ws.base = nullptr;
        g_ws.bytes = 0;
        if (e != hipSuccess) return hip_fail(e, "hipFree");
    }
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, need);
    if (e != hipSuccess || !p) {
        (void)hipGetLastError();
        return fail(EMU_ENOMEM, "hipMalloc of the workspace failed");
    }
    e = hipMemcpy(p, &status, sizeof(status), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(p);
        return hip_fail(e, "hipMemcpy(status)");
    }
    e = hipMemset((char *)p + sizeof(status), 0, HDR - sizeof(status));
    if (e != hipSuccess) {
        (void)hipFree(p);
        return hip_fail(e, "hipMemset(header)");
    }
    g_ws.base = (char *)p;
    g_ws.bytes = need;
    return EMU_OK;
}

// Phase profiling: a fixed pool of event triples, created by emu_profile_enable.
struct Profile {
    bool on = false;
    std::vector<hipEvent_t> ev;     // 3 per call
    size_t used = 0;                // triples used since the last read
} g_prof;

constexpr size_t PROFILE_CALLS = 4096;

// Event slot of the current call's phase boundary p (0, 1, 2), or null.
hipEvent_t prof_event(int p) {
    if (!g_prof.on || g_prof.used >= PROFILE_CALLS) return nullptr;
    return g_prof.ev[3 * g_prof.used + p];
}

void prof_mark(int p) {
    hipEvent_t e = prof_event(p);
    if (e) (void)hipEventRecord(e, g_stream);
    if (e && p == 2) ++g_prof.used;
}

// Areas of a workspace (the growing one, or the fixed scratch of the
// allocation-free entry point) starting at base.
unsigned *ws_status(char *base) { return reinterpret_cast<unsigned *>(base); }
F64SplitState *ws_states(char *base) { return reinterpret_cast<F64SplitState *>(base + 128); }
uint16_t *ws_planes(char *base, size_t off) { return reinterpret_cast<uint16_t *>(base + HDR + off); }
unsigned *ws_status() { return ws_status(g_ws.base); }
F64SplitState *ws_states() { return ws_states(g_ws.base); }
uint16_t *ws_planes(size_t off) { return ws_planes(g_ws.base, off); }

// Scale-aware split scratch after the planes (256-byte aligned): 64-bit maxima
// for the nA rows of A and the nB columns of B, then their int32 exponents.
struct ScaleArea {
    unsigned long long *mb;   // [nA + nB]
    int *sa, *sb;             // [nA], [nB]
};
size_t scale_bytes(int64_t nA, int64_t nB) { return 256 + (size_t)(nA + nB) * 12; }
ScaleArea ws_scales(char *base, size_t planes_bytes, int64_t nA, int64_t nB) {
    const size_t off = (HDR + planes_bytes + 255) / 256 * 256;
    ScaleArea a;
    a.mb = reinterpret_cast<unsigned long long *>(base + off);
    a.sa = reinterpret_cast<int *>(a.mb + nA + nB);
    a.sb = a.sa + nA;
    return a;
}
ScaleArea ws_scales(size_t planes_bytes, int64_t nA, int64_t nB) {
    return ws_scales(g_ws.base, planes_bytes, nA, nB);
}

// ---------------------------------------------------------------------------
// The fixed scratch of emu_dgemm_noalloc (defined at file scope, above).
constexpr int MAX_DEVICES = 64;
char *g_scratch_ptr[MAX_DEVICES] = {};

// The current device's scratch address (set up on the device's first call:
// the symbol lookup and a clear of the status word, a kernel rather than a
// memset so that a captured first call records nothing else), or null with
// *rc set.
char *scratch_for_current_device(int *rc) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        *rc = hip_fail(e, "hipGetDevice");
        return nullptr;
    }
    if (dev < 0 || dev >= MAX_DEVICES) {
        *rc = fail(EMU_EINVAL, "device index beyond the allocation-free entry point's table");
        return nullptr;
    }
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) {
            *rc = hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
            return nullptr;
        }
        e = launch_fill_f32(reinterpret_cast<float *>(ptr), 1, 1, 1, g_stream);
        if (e != hipSuccess) {
            *rc = hip_fail(e, "clear of the scratch status word");
            return nullptr;
        }
        g_scratch_ptr[dev] = static_cast<char *>(ptr);
    }
    return g_scratch_ptr[dev];
}

// Depth d of the triangular selection S_d = {(i, j) : i, j < 6, i + j < d}
// (Eq. product-selection) with N_p(d) = |S_d| = nprod, or -1.
int nprod_to_d(int nprod) {
    static const int count[12] = {0, 1, 3, 6, 10, 15, 21, 26, 30, 33, 35, 36};
    for (int d = 1; d <= 11; ++d)
        if (count[d] == nprod) return d;
    return -1;
}

// Validation shared by both GEMMs (Sec. 3.2 problem statement, row-major, with
// the BLAS transposition flags: op(A) is M x K, op(B) is K x N).
int trans_flag(char t, bool *tr) {
    switch (t) {
        case 'N': case 'n': *tr = false; return EMU_OK;
        case 'T': case 't': case 'C': case 'c': *tr = true; return EMU_OK;
        default: return fail(EMU_EINVAL, "transa / transb must be 'N' or 'T'");
    }
}

int check_gemm_args(bool ta, bool tb, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                    const void *B, int64_t ldb, const void *C, int64_t ldc, bool need_ab) {
    if (M < 0 || N < 0 || K < 0) return fail(EMU_EINVAL, "M, N and K must be non-negative");
    const int64_t acols = ta ? M : K, bcols = tb ? K : N;
    if (lda < (acols > 1 ? acols : 1)) return fail(EMU_EINVAL, ta ? "lda < max(1, M)" : "lda < max(1, K)");
    if (ldb < (bcols > 1 ? bcols : 1)) return fail(EMU_EINVAL, tb ? "ldb < max(1, K)" : "ldb < max(1, N)");
    if (ldc < (N > 1 ? N : 1)) return fail(EMU_EINVAL, "ldc < max(1, N)");
    if (M > 0 && N > 0 && !C) return fail(EMU_EINVAL, "C is NULL");
    if (need_ab && M > 0 && N > 0 && K > 0 && (!A || !B)) return fail(EMU_EINVAL, "A or B is NULL");
    if (M > (int64_t)1 << 31 || N > (int64_t)1 << 31 || K > (int64_t)1 << 36)
        return fail(EMU_EINVAL, "matrix dimension too large");
    return EMU_OK;
}

struct Shape {
    int64_t KB, RpadA, RpadB;
    size_t bytesA, bytesB;
};

// Packed sizes: rows padded to whole GEMM tiles (tile_m, tile_n are multiples
// of ROW_GROUP), reduction padded to whole k-blocks.
Shape plan(int64_t M, int64_t N, int64_t K, int nplanes, int64_t tile_m, int64_t tile_n,
           int64_t KB = 0) {
    Shape s;
    s.KB = KB > 0 ? KB : (K + KBLK - 1) / KBLK;
    s.RpadA = round_up(M, tile_m) + ROW_SKEW_TILES * tile_m;
    s.RpadB = round_up(N, tile_n) + ROW_SKEW_TILES * tile_n;
    s.bytesA = (size_t)nplanes * plane_elems(s.KB, s.RpadA) * 2;
    s.bytesB = (size_t)nplanes * plane_elems(s.KB, s.RpadB) * 2;
    return s;
}

}  // namespace

extern "C" {

int emu_set_stream(void *hip_stream) {
    const hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    if (s != g_stream && g_ws.base) {
        // Every call shares the one workspace: work queued on the new stream
        // must not start before the calls already queued on the old one are
        // done with it.  An event dependency, no host synchronisation.
        if (!g_switch_event) {
            hipError_t e = hipEventCreateWithFlags(&g_switch_event, hipEventDisableTiming);
            if (e != hipSuccess) {
                g_switch_event = nullptr;
                return hip_fail(e, "hipEventCreateWithFlags");
            }
        }
        hipError_t e = hipEventRecord(g_switch_event, g_stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(s, g_switch_event, 0);
        if (e != hipSuccess) return hip_fail(e, "stream switch");
    }
    g_stream = s;
    return EMU_OK;
}

int emu_set_split_mode(int mode) {
    if (mode != EMU_SPLIT_SYM && mode != EMU_SPLIT_LITERAL)
        return fail(EMU_EINVAL, "split mode must be EMU_SPLIT_SYM or EMU_SPLIT_LITERAL");
    g_split_mode = mode;
    return EMU_OK;
}

int emu_set_fallback(int mode) {
    if (mode != EMU_FALLBACK_NONE && mode != EMU_FALLBACK_FP64)
        return fail(EMU_EINVAL, "fallback must be EMU_FALLBACK_NONE or EMU_FALLBACK_FP64");
    g_fallback = mode;
    return EMU_OK;
}

int emu_set_sgemm_split(int mode) {
    if (mode != EMU_SGEMM_SPLIT_PASS && mode != EMU_SGEMM_SPLIT_STREAMED)
        return fail(EMU_EINVAL, "mode must be EMU_SGEMM_SPLIT_PASS or EMU_SGEMM_SPLIT_STREAMED");
    g_sgemm_split = mode;
    return EMU_OK;
}

int emu_set_split_scope(int scope) {
    if (scope != EMU_SCOPE_OPERAND && scope != EMU_SCOPE_ROWCOL && scope != EMU_SCOPE_KBIN)
        return fail(EMU_EINVAL,
                    "split scope must be EMU_SCOPE_OPERAND, EMU_SCOPE_ROWCOL or EMU_SCOPE_KBIN");
    g_split_scope = scope;
    return EMU_OK;
}

const char *emu_last_error(void) { return g_err.c_str(); }

int64_t emu_workspace_bytes(void) { return (int64_t)g_ws.bytes; }

int emu_release_workspace(void) {
    if (!g_ws.base) return EMU_OK;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    e = hipFree(g_ws.base);
    g_ws.base = nullptr;
    g_ws.bytes = 0;
    if (e != hipSuccess) return hip_fail(e, "hipFree");
    return EMU_OK;
}

int emu_profile_enable(int on) {
    if (on && !g_prof.on) {
        g_prof.ev.assign(3 * PROFILE_CALLS, nullptr);
        for (auto &e : g_prof.ev) {
            hipError_t r = hipEventCreate(&e);
            if (r != hipSuccess) return hip_fail(r, "hipEventCreate");
        }
        g_prof.used = 0;
        g_prof.on = true;
    } else if (!on && g_prof.on) {
        (void)hipDeviceSynchronize();
        for (auto &e : g_prof.ev)
            if (e) (void)hipEventDestroy(e);
        g_prof.ev.clear();
        g_prof.used = 0;
        g_prof.on = false;
    }
    return EMU_OK;
}

int emu_profile_read(int64_t cap, double *split_ms, double *gemm_ms, int64_t *calls) {
    if (!calls || (cap > 0 && (!split_ms || !gemm_ms)))
        return fail(EMU_EINVAL, "NULL output pointer");
    *calls = 0;
    if (!g_prof.on) return EMU_OK;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    for (size_t i = 0; i < g_prof.used && (int64_t)i < cap; ++i) {
        float a = 0.f, b = 0.f;
        e = hipEventElapsedTime(&a, g_prof.ev[3 * i], g_prof.ev[3 * i + 1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        e = hipEventElapsedTime(&b, g_prof.ev[3 * i + 1], g_prof.ev[3 * i + 2]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        split_ms[i] = a;
        gemm_ms[i] = b;
    }
    *calls = (int64_t)g_prof.used;
    g_prof.used = 0;
    return EMU_OK;
}

int emu_domain_status(unsigned *flags) {
    if (!flags) return fail(EMU_EINVAL, "flags is NULL");
    *flags = 0;
    // the status words of the workspace and of the current device's scratch
    int dev = 0;
    char *words[2] = {g_ws.base, nullptr};
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < MAX_DEVICES)
        words[1] = g_scratch_ptr[dev];
    if (!words[0] && !words[1]) return EMU_OK;
    hipError_t e = hipStreamSynchronize(g_stream);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    for (char *w : words) {
        if (!w) continue;
        unsigned f = 0;
        e = hipMemcpy(&f, w, sizeof(unsigned), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy(status)");
        *flags |= f;
        const unsigned zero = 0;
        e = hipMemcpy(w, &zero, sizeof(unsigned), hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy(status)");
    }
    return EMU_OK;
}

int emu_sgemm_ex(char transa, char transb, int64_t M, int64_t N, int64_t K, float alpha,
                 const float *A, int64_t lda, const float *B, int64_t ldb, float beta, float *C,
                 int64_t ldc) {
    bool ta = false, tb = false;
    int rc = trans_flag(transa, &ta);
    if (!rc) rc = trans_flag(transb, &tb);
    if (!rc) rc = check_gemm_args(ta, tb, M, N, K, A, lda, B, ldb, C, ldc, alpha != 0.0f);
    if (rc) return rc;
    g_err.clear();
    if (M == 0 || N == 0) return EMU_OK;
    if (K == 0 || alpha == 0.0f) {
        hipError_t e = launch_scale_c_f32(C, M, N, ldc, beta, g_stream);
        return e == hipSuccess ? EMU_OK : hip_fail(e, "scale C");
    }
    if (g_sgemm_split == EMU_SGEMM_SPLIT_STREAMED) {
        // the product kernel splits the operands itself (128-row tiles)
        const int splits = sgemm_splits(M, N, (K + KBLK - 1) / KBLK, 128);
        const size_t part_bytes = splits > 1 ? (size_t)splits * M * N * sizeof(float) : 0;
        rc = ensure_workspace(part_bytes > 0 ? part_bytes : 1);
        if (rc) return rc;
        float *part = splits > 1 ? reinterpret_cast<float *>(ws_planes(0)) : nullptr;
        prof_mark(0);
        prof_mark(1);
        hipError_t e = launch_gemm_f32_streamed(A, lda, ta, B, ldb, tb, C, M, N, K, ldc, alpha,
                                                beta, splits, part, ws_status(), g_stream);
        if (e != hipSuccess) return hip_fail(e, "gemm_f32_streamed");
        prof_mark(2);
        return EMU_OK;
    }
    const int tile_m = sgemm_tile_m(M, N, (K + KBLK - 1) / KBLK);
    const Shape s = plan(M, N, K, 3, tile_m, SGEMM_NT);
    // few output tiles: split the reduction (partial sums after the planes)
    const int splits = sgemm_splits(M, N, s.KB, tile_m);
    const size_t part_off = (s.bytesA + s.bytesB + 255) / 256 * 256;
    const size_t part_bytes = splits > 1 ? (size_t)splits * M * N * sizeof(float) : 0;
    rc = ensure_workspace(part_off + part_bytes);
    if (rc) return rc;
    uint16_t *Ap = ws_planes(0), *Bp = ws_planes(s.bytesA);
    float *part = splits > 1 ? reinterpret_cast<float *>(ws_planes(part_off)) : nullptr;
    prof_mark(0);
    // op(A) rows are A's rows ('N') or A's columns ('T': A is K x M, packed as a
    // B operand); op(B) columns likewise; both operands in one launch
    const F32SplitOperand ops[2] = {
        {A, ta ? K : M, ta ? M : K, lda, ta ? 1 : 0, Ap, s.RpadA},
        {B, tb ? N : K, tb ? K : N, ldb, tb ? 0 : 1, Bp, s.RpadB}};
    hipError_t e = launch_split_f32(ops, 2, s.KB, ws_status(), g_stream);
    if (e != hipSuccess) return hip_fail(e, "split_f32");
    prof_mark(1);
    e = launch_gemm_f32(Ap, Bp, C, M, N, s.KB, s.RpadA, s.RpadB, ldc, alpha, beta, tile_m, splits,
                        part, g_stream);
    if (e != hipSuccess) return hip_fail(e, "gemm_f32");
    prof_mark(2);
    return EMU_OK;
}

int emu_sgemm(int64_t M, int64_t N, int64_t K, const float *A, int64_t lda, const float *B,
              int64_t ldb, float *C, int64_t ldc) {
    return emu_sgemm_ex('N', 'N', M, N, K, 1.0f, A, lda, B, ldb, 0.0f, C, ldc);
}

}  // extern "C"

namespace {

// Bytes of workspace (after the header) an emulated DGEMM of depth d needs.
// How one emulated DGEMM runs: with the row/column weights of the scale-aware
// split, and with the native FP64 fallback armed.
struct DgemmOpts {
    bool scaled;
    bool fallback;
};

DgemmOpts current_opts() {
    return {g_split_scope != EMU_SCOPE_OPERAND, g_fallback == EMU_FALLBACK_FP64};
}

// Workspace areas of one emulated DGEMM after the header: packed planes, then
// (256-byte aligned) the weights of the scale-aware split, then a copy of C
// for a fallback that must still read beta C.
struct DgemmLayout {
    Shape s;
    size_t scale_off, csave_off, bytes;
};

DgemmLayout dgemm_layout(int64_t M, int64_t N, int64_t K, int d, DgemmOpts o, double beta) {
    DgemmLayout L;
    // the DGEMM kernel's tile rows and k-block multiple (padding is zero)
    const int64_t KB = (K + KBLK - 1) / KBLK;
    L.s = plan(M, N, K, dgemm_planes(d), dgemm_tile_rows(d, M, N, KB), DGEMM_NT,
               dgemm_kb_padded(d, M, N, KB));
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    L.scale_off = up(L.s.bytesA + L.s.bytesB);
    L.csave_off = up(L.scale_off + (o.scaled ? scale_bytes(M, N) : 0));
    L.bytes = L.csave_off + ((o.fallback && beta != 0.0) ? (size_t)M * N * sizeof(double) : 0);
    return L;
}

// The accumulated status word (offset 0 of a workspace header) and the word of
// the current call (offset 64) that an armed fallback reads.
unsigned *ws_call_status(char *base) { return reinterpret_cast<unsigned *>(base + 64); }

// The emulated DGEMM on a workspace at base (header, planes, weights), after
// argument validation; M, N, K > 0 and alpha != 0.  status_to: the word the
// split's flags go to when the fallback is not armed (null: the accumulated
// word).
int dgemm_run(char *base, DgemmOpts o, bool ta, bool tb, int64_t M, int64_t N, int64_t K,
              double alpha, const double *A, int64_t lda, const double *B, int64_t ldb,
              double beta, double *C, int64_t ldc, int d, unsigned *status_to = nullptr) {
    // Only the slices the retained products read are materialised; the levels
    // after them never influence the earlier slices.
    const int np = dgemm_planes(d);
    const DgemmLayout L = dgemm_layout(M, N, K, d, o, beta);
    const Shape &s = L.s;
    uint16_t *Ap = ws_planes(base, 0), *Bp = ws_planes(base, s.bytesA);
    F64SplitState *st = ws_states(base);
    const ScaleArea sc = ws_scales(base, L.scale_off, M, N);
    double *Csave = reinterpret_cast<double *>(base + HDR + L.csave_off);
    // stored shapes: A is M x K ('N') or K x M ('T'); B is K x N ('N') or N x K ('T')
    const int64_t ar = ta ? K : M, ac = ta ? M : K, br = tb ? N : K, bc = tb ? K : N;
    prof_mark(0);
    hipError_t e = hipSuccess;
    // an armed fallback reads the flags of this call alone: they go to the
    // call's own word (cleared by a kernel, not a memset), and the fallback
    // kernel adds them to the accumulated word
    unsigned *split_status =
        o.fallback ? ws_call_status(base) : (status_to ? status_to : ws_status(base));
    if (o.fallback) {
        e = launch_fill_f32(reinterpret_cast<float *>(split_status), 1, 1, 1, g_stream);
        if (e != hipSuccess) return hip_fail(e, "clear call status");
    }
    if (o.scaled) {
        // weights: rows of op(A), columns of op(B) (the scale-aware split)
        e = launch_scale_exponents(A, ar, ac, lda, ta, sc.mb, sc.sa, g_stream);
        if (e != hipSuccess) return hip_fail(e, "scale_exponents(A)");
        e = launch_scale_exponents(B, br, bc, ldb, !tb, sc.mb + M, sc.sb, g_stream);
        if (e != hipSuccess) return hip_fail(e, "scale_exponents(B)");
    }
    // both operands in one launch per phase: op(A)'s rows are A's rows ('N') or
    // A's columns ('T', packed as a B operand), op(B)'s columns likewise
    const F64SplitOperand ops[2] = {
        {A, ar, ac, lda, ta ? 1 : 0, o.scaled ? sc.sa : nullptr, Ap, s.RpadA, st},
        {B, br, bc, ldb, tb ? 0 : 1, o.scaled ? sc.sb : nullptr, Bp, s.RpadB, st + F64_SLOTS}};
    e = launch_split_f64(ops, 2, s.KB, np, g_split_mode, d, split_status, g_stream);
    if (e != hipSuccess) return hip_fail(e, "split_f64");
    prof_mark(1);
    const bool save_c = o.fallback && beta != 0.0;
    if (save_c) {
        e = launch_copy_matrix_f64(C, ldc, Csave, N, M, N, g_stream);
        if (e != hipSuccess) return hip_fail(e, "save C");
    }
    e = launch_gemm_f64(Ap, Bp, C, M, N, s.KB, s.RpadA, s.RpadB, ldc, o.scaled ? sc.sa : nullptr,
                        o.scaled ? sc.sb : nullptr, alpha, beta, d, g_stream);
    if (e != hipSuccess) return hip_fail(e, "gemm_f64");
    if (o.fallback) {
        e = launch_fallback_dgemm(split_status, ws_status(base), M, N, K, alpha, A, lda, ta, B, ldb,
                                  tb, beta, save_c ? Csave : C, save_c ? N : ldc, C, ldc, g_stream);
        if (e != hipSuccess) return hip_fail(e, "fallback_dgemm");
    }
    prof_mark(2);
    return EMU_OK;
}

std::vector<int> g_kbin_idx;   // host copy of the K-binned index lists

// The K-binned scope: classes of the reduction indices on the device, one
// stream synchronisation to read them, then for every class in ascending
// order the gather of its columns of op(A) and rows of op(B) and a row/column
// scaled emulated DGEMM of the group, added in FP64 to the previous groups'
// sum (the first group stores, the others use the beta = 1 update, which adds
// fl(P_g + S)); the BLAS update alpha S + beta C follows unless alpha = 1 and
// beta = 0 (then the groups accumulate in C itself).  An armed fallback reads
// the flags of all groups and replaces the whole result.
int dgemm_kbin(bool ta, bool tb, int64_t M, int64_t N, int64_t K, double alpha, const double *A,
               int64_t lda, const double *B, int64_t ldb, double beta, double *C, int64_t ldc,
               int d) {
    const bool fb = g_fallback == EMU_FALLBACK_FP64;
    const bool direct = alpha == 1.0 && beta == 0.0;
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    // workspace after the area of the largest group's DGEMM (its planes and weights)
    size_t off = up(dgemm_layout(M, N, K, d, {true, false}, 0.0).bytes);
    const int64_t MN = M > N ? M : N;
    const size_t o_sa = off;  off = up(off + (size_t)M * 4);
    const size_t o_sb = off;  off = up(off + (size_t)N * 4);
    const size_t o_mx = off;  off = up(off + (size_t)MN * 8);
    const size_t o_ma = off;  off = up(off + (size_t)K * 8);
    const size_t o_mb = off;  off = up(off + (size_t)K * 8);
    const size_t o_cl = off;  off = up(off + (size_t)K * 4);
    const size_t o_ix = off;  off = up(off + (size_t)K * 4);
    const size_t o_ga = off;  off = up(off + (size_t)M * K * 8);
    const size_t o_gb = off;  off = up(off + (size_t)K * N * 8);
    const size_t o_p = off;   off = up(off + (direct ? 0 : (size_t)M * N * 8));
    int rc = ensure_workspace(off);
    if (rc) return rc;
    char *base = g_ws.base, *w = g_ws.base + HDR;
    int *sa = reinterpret_cast<int *>(w + o_sa), *sb = reinterpret_cast<int *>(w + o_sb);
    auto *mx = reinterpret_cast<unsigned long long *>(w + o_mx);
    auto *ma = reinterpret_cast<unsigned long long *>(w + o_ma);
    auto *mb = reinterpret_cast<unsigned long long *>(w + o_mb);
    int *cls = reinterpret_cast<int *>(w + o_cl), *idx = reinterpret_cast<int *>(w + o_ix);
    double *GA = reinterpret_cast<double *>(w + o_ga), *GB = reinterpret_cast<double *>(w + o_gb);
    double *P = reinterpret_cast<double *>(w + o_p);
    unsigned *acc_st = ws_status(base), *call_st = ws_call_status(base);
    const int64_t ar = ta ? K : M, ac = ta ? M : K, br = tb ? N : K, bc = tb ? K : N;
    hipError_t e = hipSuccess;
    if (fb) {
        e = launch_fill_f32(reinterpret_cast<float *>(call_st), 1, 1, 1, g_stream);
        if (e != hipSuccess) return hip_fail(e, "clear call status");
    }
    e = launch_scale_exponents(A, ar, ac, lda, ta, mx, sa, g_stream);
    if (e == hipSuccess) e = launch_scale_exponents(B, br, bc, ldb, !tb, mx, sb, g_stream);
    if (e == hipSuccess)
        e = launch_kbin_classes(A, lda, ta, B, ldb, tb, M, N, K, sa, sb, ma, mb, KBIN_WIDTH,
                                KBIN_MAX, cls, g_stream);
    if (e != hipSuccess) return hip_fail(e, "kbin classes");
    std::vector<int> h((size_t)K);
    e = hipMemcpyAsync(h.data(), cls, (size_t)K * 4, hipMemcpyDeviceToHost, g_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(g_stream);
    if (e != hipSuccess) return hip_fail(e, "kbin classes to the host");
    // the index lists stay alive in g_kbin_idx until the next call, which
    // synchronises the stream before it rewrites them
    std::vector<int> &ks = g_kbin_idx;
    ks.clear();
    std::vector<std::pair<size_t, int64_t>> groups;   // (first index in ks, size)
    for (int c = 0; c < KBIN_MAX; ++c) {
        const size_t first = ks.size();
        for (int64_t k = 0; k < K; ++k)
            if (h[(size_t)k] == c) ks.push_back((int)k);
        if (ks.size() > first) groups.emplace_back(first, (int64_t)(ks.size() - first));
    }
    if (groups.empty()) {   // every product term is an exact zero
        e = launch_scale_c_f64(C, M, N, ldc, beta, g_stream);
        return e == hipSuccess ? EMU_OK : hip_fail(e, "scale C");
    }
    e = hipMemcpyAsync(idx, ks.data(), ks.size() * 4, hipMemcpyHostToDevice, g_stream);
    if (e != hipSuccess) return hip_fail(e, "kbin index upload");
    double *T = direct ? C : P;
    const int64_t ldt = direct ? ldc : N;
    for (size_t g = 0; g < groups.size(); ++g) {
        const int64_t kb = groups[g].second;
        e = launch_kbin_gather(A, lda, ta, B, ldb, tb, M, N, idx + groups[g].first, kb, GA, GB,
                               g_stream);
        if (e != hipSuccess) return hip_fail(e, "kbin gather");
        rc = dgemm_run(base, {true, false}, false, false, M, N, kb, 1.0, GA, kb, GB, N,
                       g == 0 ? 0.0 : 1.0, T, ldt, d, fb ? call_st : acc_st);
        if (rc) return rc;
    }
    if (fb) {
        // C is untouched unless direct (then beta = 0 and C is not read)
        e = launch_fallback_dgemm(call_st, acc_st, M, N, K, alpha, A, lda, ta, B, ldb, tb, beta,
                                  C, ldc, C, ldc, g_stream);
        if (e != hipSuccess) return hip_fail(e, "fallback_dgemm");
    }
    if (!direct) {
        e = launch_axpby_f64(P, N, C, ldc, M, N, alpha, beta, fb ? call_st : nullptr, g_stream);
        if (e != hipSuccess) return hip_fail(e, "alpha P + beta C");
    }
    return EMU_OK;
}

// Validation and the degenerate cases of the DGEMM entry points; returns 1 when
// dgemm_run must follow (d and the transposition flags set), else the result.
int dgemm_prologue(char transa, char transb, int64_t M, int64_t N, int64_t K, double alpha,
                   const double *A, int64_t lda, const double *B, int64_t ldb, double beta,
                   double *C, int64_t ldc, int nprod, int *d, bool *ta, bool *tb, int *rc) {
    *d = nprod_to_d(nprod);
    if (*d < 0) {
        *rc = fail(EMU_EINVAL, "nprod must be 1, 3, 6, 10, 15, 21, 26, 30, 33, 35 or 36");
        return 0;
    }
    *rc = trans_flag(transa, ta);
    if (!*rc) *rc = trans_flag(transb, tb);
    if (!*rc) *rc = check_gemm_args(*ta, *tb, M, N, K, A, lda, B, ldb, C, ldc, alpha != 0.0);
    if (*rc) return 0;
    g_err.clear();
    if (M == 0 || N == 0) return 0;
    if (K == 0 || alpha == 0.0) {
        hipError_t e = launch_scale_c_f64(C, M, N, ldc, beta, g_stream);
        *rc = e == hipSuccess ? EMU_OK : hip_fail(e, "scale C");
        return 0;
    }
    return 1;
}

}  // namespace

extern "C" {

int emu_dgemm_ex(char transa, char transb, int64_t M, int64_t N, int64_t K, double alpha,
                 const double *A, int64_t lda, const double *B, int64_t ldb, double beta,
                 double *C, int64_t ldc, int nprod) {
    int d = 0, rc = EMU_OK;
    bool ta = false, tb = false;
    if (!dgemm_prologue(transa, transb, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, nprod, &d,
                        &ta, &tb, &rc))
        return rc;
    if (g_split_scope == EMU_SCOPE_KBIN)
        return dgemm_kbin(ta, tb, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, d);
    const DgemmOpts o = current_opts();
    rc = ensure_workspace(dgemm_layout(M, N, K, d, o, beta).bytes);
    if (rc) return rc;
    return dgemm_run(g_ws.base, o, ta, tb, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, d);
}

int emu_dgemm_noalloc(int64_t M, int64_t N, int64_t K, const double *A, int64_t lda,
                      const double *B, int64_t ldb, double *C, int64_t ldc, int nprod) {
    int d = 0, rc = EMU_OK;
    bool ta = false, tb = false;
    if (!dgemm_prologue('N', 'N', M, N, K, 1.0, A, lda, B, ldb, 0.0, C, ldc, nprod, &d, &ta, &tb,
                        &rc))
        return rc;
    if (g_split_scope == EMU_SCOPE_KBIN)
        return fail(EMU_EINVAL, "emu_dgemm_noalloc: the K-binned scope needs the growing workspace");
    const DgemmOpts o = current_opts();
    const size_t need = HDR + dgemm_layout(M, N, K, d, o, 0.0).bytes;
    if (need > NOALLOC_BYTES) {
        g_err = "emu_dgemm_noalloc: this problem needs " + std::to_string(need) +
                " bytes of scratch, more than the fixed " + std::to_string(NOALLOC_BYTES);
        return EMU_ENOMEM;
    }
    char *base = scratch_for_current_device(&rc);
    if (!base) return rc;
    return dgemm_run(base, o, false, false, M, N, K, 1.0, A, lda, B, ldb, 0.0, C, ldc, d);
}

int emu_dgemm(int64_t M, int64_t N, int64_t K, const double *A, int64_t lda, const double *B,
              int64_t ldb, double *C, int64_t ldc, int nprod) {
    return emu_dgemm_ex('N', 'N', M, N, K, 1.0, A, lda, B, ldb, 0.0, C, ldc, nprod);
}

static int check_split_args(int64_t R, int64_t Cc, const void *X, int64_t ldx, int as_b,
                            const void *out) {
    if (R < 0 || Cc < 0) return fail(EMU_EINVAL, "R and Cc must be non-negative");
    if (ldx < (Cc > 1 ? Cc : 1)) return fail(EMU_EINVAL, "ldx < max(1, Cc)");
    if (as_b != 0 && as_b != 1) return fail(EMU_EINVAL, "as_b must be 0 or 1");
    if (R > 0 && Cc > 0 && (!X || !out)) return fail(EMU_EINVAL, "NULL pointer");
    return EMU_OK;
}

int emu_split_f32(int64_t R, int64_t Cc, const float *X, int64_t ldx, int as_b, uint16_t *comps) {
    int rc = check_split_args(R, Cc, X, ldx, as_b, comps);
    if (rc) return rc;
    g_err.clear();
    if (R == 0 || Cc == 0) return EMU_OK;
    const int64_t rows = as_b ? Cc : R, K = as_b ? R : Cc;   // packed rows and reduction length
    const Shape s = plan(rows, 1, K, 3, ROW_GROUP, ROW_GROUP);
    rc = ensure_workspace(s.bytesA);
    if (rc) return rc;
    uint16_t *P = ws_planes(0);
    const F32SplitOperand op = {X, R, Cc, ldx, as_b != 0 ? 1 : 0, P, s.RpadA};
    hipError_t e = launch_split_f32(&op, 1, s.KB, ws_status(), g_stream);
    if (e != hipSuccess) return hip_fail(e, "split_f32");
    e = launch_unpack(P, 3, s.KB, s.RpadA, R, Cc, as_b != 0, comps, g_stream);
    if (e != hipSuccess) return hip_fail(e, "unpack");
    return EMU_OK;
}

int emu_split_f64(int64_t R, int64_t Cc, const double *X, int64_t ldx, int as_b,
                  uint16_t *slices, int32_t *v) {
    int rc = check_split_args(R, Cc, X, ldx, as_b, slices);
    if (rc) return rc;
    if (!v) return fail(EMU_EINVAL, "v is NULL");
    g_err.clear();
    const int64_t rows = as_b ? Cc : R, K = as_b ? R : Cc;
    const Shape s = plan(rows, 1, K, 6, ROW_GROUP, ROW_GROUP);
    const bool scaled = g_split_scope != EMU_SCOPE_OPERAND;   // KBIN splits as ROWCOL here
    rc = ensure_workspace((s.bytesA > 0 ? s.bytesA : 1) + (scaled ? scale_bytes(rows, 0) : 0));
    if (rc) return rc;
    uint16_t *P = ws_planes(0);
    F64SplitState *st = ws_states();
    const ScaleArea sc = ws_scales(s.bytesA > 0 ? s.bytesA : 1, rows, 0);
    hipError_t e = hipSuccess;
    if (scaled) {
        e = launch_scale_exponents(X, R, Cc, ldx, as_b != 0, sc.mb, sc.sa, g_stream);
        if (e != hipSuccess) return hip_fail(e, "scale_exponents");
    }
    const F64SplitOperand op = {X, R, Cc, ldx, as_b != 0 ? 1 : 0, scaled ? sc.sa : nullptr, P,
                                s.RpadA, st};
    e = launch_split_f64(&op, 1, s.KB, 6, g_split_mode, 0, ws_status(), g_stream);
    if (e != hipSuccess) return hip_fail(e, "split_f64");
    if (R > 0 && Cc > 0) {
        e = launch_unpack(P, 6, s.KB, s.RpadA, R, Cc, as_b != 0, slices, g_stream);
        if (e != hipSuccess) return hip_fail(e, "unpack");
    }
    e = launch_copy_v(st, v, g_stream);
    if (e != hipSuccess) return hip_fail(e, "copy_v");
    return EMU_OK;
}

int emu_scale_exponents(int64_t R, int64_t Cc, const double *X, int64_t ldx, int by_col,
                        int32_t *s) {
    if (R < 0 || Cc < 0) return fail(EMU_EINVAL, "R and Cc must be non-negative");
    if (ldx < (Cc > 1 ? Cc : 1)) return fail(EMU_EINVAL, "ldx < max(1, Cc)");
    if (by_col != 0 && by_col != 1) return fail(EMU_EINVAL, "by_col must be 0 or 1");
    const int64_t n = by_col ? Cc : R;
    if (n > 0 && (!s || (R > 0 && Cc > 0 && !X))) return fail(EMU_EINVAL, "NULL pointer");
    g_err.clear();
    if (n == 0) return EMU_OK;
    int rc = ensure_workspace(scale_bytes(n, 0));
    if (rc) return rc;
    const ScaleArea sc = ws_scales(0, n, 0);
    hipError_t e;
    if (R == 0 || Cc == 0) {
        e = launch_fill_f32(reinterpret_cast<float *>(s), 1, n, n, g_stream);   // no entries: 0
    } else {
        e = launch_scale_exponents(X, R, Cc, ldx, by_col != 0, sc.mb, s, g_stream);
    }
    return e == hipSuccess ? EMU_OK : hip_fail(e, "scale_exponents");
}

}  // extern "C"
