#!/usr/bin/env python3
"""Benchmark of FP32/FP64 GEMM emulated through BF16 component products on
one MI355X: effective TFLOP/s (2MNK / t) of emu-SGEMM and emu-DGEMM for every
product count, with the bf16 MFMA roofline fraction of the product GEMMs.

One step = one pass of the whole hot path at M = N = K = 8192:
  emu_sgemm (3 BF16 components, 6 products; standard-normal FP32 inputs), then
  emu_dgemm with nprod = 6, 10, 15, 21 (six-slice split; wide-range FP64 inputs
  s * m * 2^e, m uniform in [1, 2), e uniform integer in [-20, 20]).
Each call includes its split/pack kernels, its GEMM kernel and its FP64
reconstruction, exactly as the library runs them; inputs are resident in HBM
before the timed region.

Prints one JSON line.  Also reported: per-variant phase times from HIP events
recorded by the library on its stream (split/pack vs GEMM, the analog of the
paper's runtime breakdown), the roofline object of the dominant kernel, a
sampled parity check against the CPU oracle, the oracle itself timed on the
host cores as a baseline, and, as context outside the step, the other product
counts of the selection sequence (nprod 1, 3 and 26 .. 36) on the same inputs.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA (AMD published)
PEAK_FP32_MATRIX = 157.3       # context: native FP32 matrix
PEAK_FP64_MATRIX = 78.6        # context: native FP64 matrix/vector
PEAK_HBM_TBS = 8.0             # MI355X HBM3E (AMD published)
TARGET_FRAC = 0.60             # bf16 MFMA fraction the product GEMMs aim for
# The paper's accuracy at m = n = k = 8192, uniform[-1, 1] inputs (Table
# accuracy, Sec. 8.2: e_F / e_scaled against oneMKL DGEMM), as printed.
PAPER_ACCURACY_8192 = {"emu-SGEMM": [3.97e-7, 4.16e-8], "emu-DGEMM-6": [1.49e-8, 1.24e-9],
                       "emu-DGEMM-10": [3.25e-11, 2.86e-12], "emu-DGEMM-15": [6.96e-14, 6.15e-15],
                       "emu-DGEMM-21": [9.41e-16, 1.52e-16]}
# The paper's own figures at m = n = k = 8192 (Figs. fullcore-fp32 and
# fullcore-fp64: 2 x Xeon Platinum 8462Y+, AMX-BF16, 64 threads, oneMKL 2026.1
# baselines), as printed; another machine, context only.
PAPER_CONTEXT_8192 = {
    "machine": "2x Intel Xeon Platinum 8462Y+ (AMX-BF16), 64 threads; values as printed in the "
               "paper's Figs. fullcore-fp32/fullcore-fp64 (axis labelled GFLOPS)",
    "emu_sgemm": 11.174, "mkl_sgemm": 9.603,
    "emu_dgemm": {"6": 6.787, "10": 4.543, "15": 3.224, "21": 2.359}, "mkl_dgemm": 4.887,
}
VARIANTS = [("sgemm", 6), ("dgemm", 6), ("dgemm", 10), ("dgemm", 15), ("dgemm", 21)]
_CSRC = "paper_2609_04663_amd/csrc/"
# sources a GEMM kernel is compiled from (a stored traffic figure is only used
# while their hash is unchanged)
KERNEL_SOURCES = {
    "sgemm": [_CSRC + "gemm_f32.hip", _CSRC + "gemm_common.h", _CSRC + "emu_internal.h"],
    "dgemm": [_CSRC + "gemm_f64.hip", _CSRC + "gemm_common.h", _CSRC + "emu_internal.h"],
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash(rels):
    h = hashlib.sha256()
    for rel in rels:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for(kernel_key):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    e = t.get(kernel_key)
    if not e:
        return None
    src = KERNEL_SOURCES[kernel_key.split(":")[0]]
    if e.get("source_sha256_16") != source_hash(src):
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(args, n, A32, B32, A64, B64, C32, C64, scope):
    """The oracle, as it stands, on the host: its split of the full operands
    (timed apart) and rows 0 .. R - 1 of C for every variant, extrapolated to
    the full call (split + n / R times the rows); also on one thread, with the
    split timed on a 256-row stripe of each operand and 64 entries of row 0 per
    variant, extrapolated the same way.  Also checks this run's rows against
    the oracle (DGEMM bit-exact, SGEMM normwise error)."""
    import oracle as O
    R = args.cpu_rows
    rows = np.repeat(np.arange(R, dtype=np.int64), n)
    cols = np.tile(np.arange(n, dtype=np.int64), R)
    threads = O.num_threads()
    log(f"bench: oracle split of the full operands and {R} row(s) per variant ({threads} threads)")

    def timed(f):
        t0 = time.perf_counter()
        out = f()
        return out, time.perf_counter() - t0

    (ca, cb), t_s32 = timed(lambda: (O.split_f32(A32)[0], O.split_f32(B32)[0]))
    orc32, t_r32 = timed(lambda: O.sgemm_entries_from_comps(ca, cb, rows, cols))
    (sa, sb), t_s64 = timed(lambda: (O.split_f64(A64)[0], O.split_f64(B64)[0]))
    if scope != 0:
        sa = sb = None                      # the row/column scope: entries re-split below
    got32 = C32[:R].cpu().numpy().ravel()
    ref = (A32[:R].astype(np.float64) @ B32.astype(np.float64)).ravel()
    parity = {"sgemm_rows_eF_gpu": float(np.linalg.norm(got32 - ref) / np.linalg.norm(ref)),
              "sgemm_rows_eF_oracle": float(np.linalg.norm(orc32 - ref) / np.linalg.norm(ref))}
    t_rows = {}
    bitexact = {}
    for p in (6, 10, 15, 21):
        if sa is None:
            (orc64, _), t = timed(lambda: O.emu_dgemm_entries(A64, B64, rows, cols, p, scope=scope))
            t = max(t - t_s64, 0.0)
        else:
            (orc64, _), t = timed(lambda: O.dgemm_entries_from_slices(sa, sb, rows, cols, p))
        t_rows[p] = t
        bitexact[str(p)] = bool(np.array_equal(C64[p][:R].cpu().numpy().ravel(), orc64))
    parity["dgemm_rows_bitexact"] = bitexact
    scale = n / R
    full = [t_s32 + t_r32 * scale] + [t_s64 + t_rows[p] * scale for p in (6, 10, 15, 21)]
    value = len(VARIANTS) * 2.0 * n ** 3 / sum(full) / 1e12

    # one thread, smaller sample
    S_ROWS, E1 = 256, 64
    O.set_num_threads(1)
    try:
        _, t1_s32 = timed(lambda: (O.split_f32(A32[:S_ROWS]), O.split_f32(B32[:S_ROWS])))
        _, t1_s64 = timed(lambda: (O.split_f64(A64[:S_ROWS]), O.split_f64(B64[:S_ROWS])))
        r1, c1 = np.zeros(E1, np.int64), np.arange(E1, dtype=np.int64)
        _, t1_r32 = timed(lambda: O.sgemm_entries_from_comps(ca, cb, r1, c1))
        t1_rows = {}
        for p in (6, 10, 15, 21):
            if sa is None:
                break
            _, t1_rows[p] = timed(lambda: O.dgemm_entries_from_slices(sa, sb, r1, c1, p))
    finally:
        O.set_num_threads(threads)
    one_core = None
    if len(t1_rows) == 4:
        ss, se = n / S_ROWS, n * n / E1
        full1 = [t1_s32 * ss + t1_r32 * se] + [t1_s64 * ss + t1_rows[p] * se for p in (6, 10, 15, 21)]
        one_core = {
            "value": round(len(VARIANTS) * 2.0 * n ** 3 / sum(full1) / 1e12, 9),
            "cores": 1,
            "sample": (f"extrapolated: the split of a {S_ROWS}-row stripe of each operand "
                       f"(x {n // S_ROWS}) and {E1} entries of row 0 per variant "
                       f"(x {n * n // E1}); {t1_s32 + t1_s64 + t1_r32 + sum(t1_rows.values()):.1f} s"),
        }
    cpu = {
        "value": round(value, 9),
        "unit": "effective TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"extrapolated to the full {n}^3 calls: the oracle's split of both full operands "
                   f"(FP32 {t_s32:.1f} s, FP64 six slices {t_s64:.1f} s, each counted once per call) "
                   f"and rows 0..{R - 1} of C ({R * n} entries) per variant "
                   f"({t_r32 + sum(t_rows.values()):.1f} s), rows scaled by {n // R}"),
        "split_s": {"fp32": round(t_s32, 3), "fp64": round(t_s64, 3)},
        "rows_s": {"sgemm": round(t_r32, 3), **{f"dgemm-{p}": round(t, 3) for p, t in t_rows.items()}},
        "full_call_s_extrapolated": [round(x, 2) for x in full],
        "one_core": one_core,
    }
    return cpu, parity


def accuracy_probe(emu, n, R):
    """Errors on uniform[-1, 1] inputs (the paper's accuracy study, Sec. 8.2):
    rows 0 .. R - 1 of C against a double-double reference, e_F and e_scaled
    (Eqs. froerror, scalederror) on those rows, next to the paper's values at
    8192 (measured there against oneMKL, over the full matrix)."""
    import torch
    import oracle as O
    import seeded_inputs as S
    log(f"bench: accuracy probe, uniform[-1,1], rows 0..{R - 1}")
    A = S.make("uniform", 9001, (n, n), np.float64)
    B = S.make("uniform", 9002, (n, n), np.float64)
    rows = np.repeat(np.arange(R, dtype=np.int64), n)
    cols = np.tile(np.arange(n, dtype=np.int64), R)
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    hi, lo = O.ref_dd_entries(A, B, rows, cols)
    absp = O.absprod_entries(A, B, rows, cols)
    out = {}
    for p in (6, 10, 15, 21):
        got = emu.dgemm(dA, dB, p)[:R].cpu().numpy().ravel()
        out[f"emu-DGEMM-{p}"] = [O.e_F(got, (hi, lo)), O.e_scaled(got, (hi, lo), absp)[0]]
    A32, B32 = A.astype(np.float32), B.astype(np.float32)
    got = emu.sgemm(dA.float(), dB.float())[:R].cpu().numpy().ravel()
    h32 = (A32[:R].astype(np.float64) @ B32.astype(np.float64)).ravel()
    abs32 = (np.abs(A32[:R].astype(np.float64)) @ np.abs(B32.astype(np.float64))).ravel()
    out["emu-SGEMM"] = [O.e_F(got, h32), O.e_scaled(got, h32, abs32)[0]]
    return {
        "rows": R, "inputs": "uniform[-1,1], FP64 (FP32: RNE-cast), seeds 9001/9002",
        "eF_escaled": {k: [float(f"{x:.3g}") for x in v] for k, v in out.items()},
        "paper_8192_eF_escaled": PAPER_ACCURACY_8192 if n == 8192 else None,
        "note": "paper: full matrix against oneMKL (its SGEMM/DGEMM error included); here: sampled "
                "rows against exact-product references",
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--size", type=int, default=8192, help="M = N = K")
    ap.add_argument("--cpu-rows", type=int, default=4,
                    help="rows of C the oracle computes per variant for the CPU baseline")
    ap.add_argument("--no-accuracy", action="store_true",
                    help="skip the accuracy probe on uniform[-1,1] inputs (paper Table accuracy)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run one plain device-to-device copy of this many MiB: the "
                         "reference kernel that scales rocprofv3 FETCH_SIZE/WRITE_SIZE readings")
    ap.add_argument("--scope", choices=("operand", "rowcol", "kbin"), default="operand",
                    help="FP64 split exponents: the paper's operand-wide chain (default), the "
                         "scale-aware row/column weights, or those with K-binned classes")
    ap.add_argument("--no-native", action="store_true",
                    help="skip timing the vendor library's native FP32/FP64 GEMM (context)")
    ap.add_argument("--no-depths", action="store_true",
                    help="skip the context timing of the other product counts (nprod 1, 3, 26..36)")
    ap.add_argument("--print-source-hash", action="store_true",
                    help="print the source hash of each GEMM kernel and exit")
    args = ap.parse_args()
    if args.print_source_hash:
        print(json.dumps({k: source_hash(v) for k, v in KERNEL_SOURCES.items()}))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus must be 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_04663_amd as emu
    import seeded_inputs as S

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    scope = {"operand": emu.SCOPE_OPERAND, "rowcol": emu.SCOPE_ROWCOL,
             "kbin": emu.SCOPE_KBIN}[args.scope]
    emu.set_split_scope(scope)
    if args.copy_calibration_mib > 0:
        nbytes = args.copy_calibration_mib << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: calibration copy of {nbytes} bytes done")
        del src, dst
    n = args.size
    log(f"bench: generating inputs M=N=K={n}")
    sa, sb = S.seeds(2)
    A32 = S.make("normal", sa, (n, n), np.float32)
    B32 = S.make("normal", sb, (n, n), np.float32)
    da, db = S.seeds(4)
    A64 = S.make("wide", da, (n, n), np.float64)
    B64 = S.make("wide", db, (n, n), np.float64)
    sha = {k: hashlib.sha256(v.tobytes()).hexdigest()
           for k, v in (("A32", A32), ("B32", B32), ("A64", A64), ("B64", B64))}
    dA32, dB32 = torch.from_numpy(A32).cuda(), torch.from_numpy(B32).cuda()
    dA64, dB64 = torch.from_numpy(A64).cuda(), torch.from_numpy(B64).cuda()
    C32 = torch.empty((n, n), dtype=torch.float32, device="cuda")
    C64 = {p: torch.empty((n, n), dtype=torch.float64, device="cuda") for p in (6, 10, 15, 21)}

    def step():
        emu.sgemm(dA32, dB32, C=C32)
        for p in (6, 10, 15, 21):
            emu.dgemm(dA64, dB64, p, C=C64[p])

    log(f"bench: warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    emu.domain_status()
    emu.profile_enable(True)
    emu.profile_read()
    torch.cuda.synchronize()
    log(f"bench: timing {args.steps} steps")
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    split_ms, gemm_ms = emu.profile_read()
    emu.profile_enable(False)
    status = emu.domain_status()
    assert len(split_ms) == len(VARIANTS) * args.steps, "profile pool too small"

    # context: the vendor library's native FP32 and FP64 GEMM on the same inputs
    native = None
    if not args.no_native:
        def lib_rate(a, b, reps):
            c = a @ b
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                c = a @ b
            e1.record()
            torch.cuda.synchronize()
            return 2.0 * n ** 3 / (e0.elapsed_time(e1) / reps * 1e-3) / 1e12
        log("bench: native FP32/FP64 GEMM (vendor library) for context")
        native = {"fp32_tflops": round(lib_rate(dA32, dB32, 3), 2),
                  "fp64_tflops": round(lib_rate(dA64, dB64, 2), 2),
                  # the headroom of the method: one plain BF16 GEMM (FP32 accumulation)
                  "bf16_tflops": round(lib_rate(dA32.to(torch.bfloat16), dB32.to(torch.bfloat16), 5), 2),
                  "library": "torch.matmul (hipBLASLt/rocBLAS), same inputs (bf16: RNE-cast)"}

    # context: the rest of the selection sequence S_d (d = 1, 2, 7 .. 11) on the
    # same FP64 inputs, one warm-up and three profiled calls each
    depths = None
    if not args.no_depths:
        log("bench: other product counts for context")
        depths = {}
        Cx = torch.empty((n, n), dtype=torch.float64, device="cuda")   # not the step's outputs
        for p in (1, 3, 26, 30, 33, 35, 36):
            emu.dgemm(dA64, dB64, p, C=Cx)
            torch.cuda.synchronize()
            emu.profile_enable(True)
            emu.profile_read()
            for _ in range(3):
                emu.dgemm(dA64, dB64, p, C=Cx)
            torch.cuda.synchronize()
            s_ms, g_ms = emu.profile_read()
            emu.profile_enable(False)
            s_m, g_m = float(np.mean(s_ms)), float(np.mean(g_ms))
            depths[str(p)] = {
                "effective_tflops": round(2.0 * n ** 3 / ((s_m + g_m) * 1e-3) / 1e12, 2),
                "split_ms": round(s_m, 4), "gemm_ms": round(g_m, 4),
                "mfma_frac": round(p * 2.0 * n ** 3 / (g_m * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
        status |= emu.domain_status()
        del Cx

    flop = 2.0 * n ** 3
    elapsed = t1 - t0
    value = len(VARIANTS) * flop * args.steps / elapsed / 1e12
    per_variant = {}
    for vi, (kind, p) in enumerate(VARIANTS):
        s = np.array(split_ms[vi::len(VARIANTS)])
        g = np.array(gemm_ms[vi::len(VARIANTS)])
        name = "emu-SGEMM" if kind == "sgemm" else f"emu-DGEMM-{p}"
        # split/pack pass, algorithmic bytes: both operands read once, their
        # BF16 planes (3, or d = 3..6 slices) written once
        in_bytes, planes = (4, 3) if kind == "sgemm" else (8, {6: 3, 10: 4, 15: 5, 21: 6}[p])
        split_bytes = (in_bytes + 2 * planes) * 2.0 * n * n
        call = s + g
        per_variant[name] = {
            "effective_tflops": round(flop / ((s.mean() + g.mean()) * 1e-3) / 1e12, 2),
            "effective_tflops_median": round(flop / (float(np.median(call)) * 1e-3) / 1e12, 2),
            "effective_tflops_best": round(flop / (float(np.min(call)) * 1e-3) / 1e12, 2),
            "call_ms_mean": round(float(call.mean()), 4),
            "call_ms_median": round(float(np.median(call)), 4),
            "call_ms_min": round(float(np.min(call)), 4),
            "split_ms": round(float(s.mean()), 4),
            "gemm_ms": round(float(g.mean()), 4),
            "split_share": round(float(s.mean() / (s.mean() + g.mean())), 4),
            "split_gbps": round(split_bytes / (s.mean() * 1e-3) / 1e9, 1),
            "mfma_frac": round(p * flop / (g.mean() * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        }
    if native:
        native["emu_sgemm_speedup_vs_native_fp32"] = round(
            per_variant["emu-SGEMM"]["effective_tflops"] / native["fp32_tflops"], 3)
        native["bf16_frac_of_peak"] = round(native["bf16_tflops"] / PEAK_BF16_TFLOPS, 4)
        native["emu_dgemm_speedup_vs_native_fp64"] = {
            str(p): round(per_variant[f"emu-DGEMM-{p}"]["effective_tflops"] / native["fp64_tflops"], 3)
            for p in (6, 10, 15, 21)}
        if depths:
            # headroom: the same GEMM kernel with one product (A_0 B_0, FP64
            # output) against the vendor bf16 GEMM, both as bf16 MFMA fractions
            native["same_kernel_nprod1_gemm_frac_of_peak"] = depths["1"]["mfma_frac"]
    # dominant kernel: the GEMM launch with the largest share of the step
    dom = max(range(len(VARIANTS)), key=lambda i: np.mean(gemm_ms[i::len(VARIANTS)]))
    kind, p = VARIANTS[dom]
    g_avg = float(np.mean(gemm_ms[dom::len(VARIANTS)]))
    achieved = p * flop / (g_avg * 1e-3) / 1e12
    kkey = f"{kind}:{p}:{n}"
    traffic = traffic_for(kkey)
    mfma_frac = achieved / PEAK_BF16_TFLOPS
    # the bound: the larger of the two roofline fractions the launch reaches,
    # MFMA flops against the bf16 peak and counter-measured HBM bytes against
    # the HBM peak (MFMA when no traffic figure matches the current source)
    hbm_frac = (traffic / (g_avg * 1e-3) / 1e12 / PEAK_HBM_TBS) if traffic else None
    bound = "hbm" if hbm_frac is not None and hbm_frac > mfma_frac else "mfma"
    roofline = {
        # long reductions of d = 3 .. 6 run gemm_f64t_kernel (whole panels)
        "kernel": ("gemm_f32_kernel" if kind == "sgemm" else
                   f"gemm_f64t_kernel<d={ {6: 3, 10: 4, 15: 5, 21: 6}[p]}>"),
        "bound": bound, "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s", "frac": round(mfma_frac, 4),
        "traffic": traffic,
        "hbm_frac": round(hbm_frac, 4) if hbm_frac is not None else None,
        "per_launch": f"{p} x 2MNK bf16 MFMA flops / mean HIP-event time of the GEMM launch",
        "target_frac": TARGET_FRAC,
        "meets_target": bool(mfma_frac >= TARGET_FRAC),
    }
    below_target = {k: v["mfma_frac"] for k, v in per_variant.items() if v["mfma_frac"] < TARGET_FRAC}

    # sampled parity of this very run against the oracle, and the oracle timing
    cpu = None
    parity = None
    if not args.no_cpu_baseline and args.cpu_rows > 0:
        cpu, parity = cpu_baseline(args, n, A32, B32, A64, B64, C32, C64, scope)

    accuracy = None
    if not args.no_accuracy:
        accuracy = accuracy_probe(emu, n, args.cpu_rows if args.cpu_rows > 0 else 1)
        status |= emu.domain_status()

    line = {
        "metric": "effective TFLOP/s (2MNK/t) emu-SGEMM & emu-DGEMM per nprod; % bf16 MFMA peak",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"M=N=K={n}: emu-SGEMM (3 comps, 6 products, standard-normal FP32) + "
                         f"emu-DGEMM nprod 6/10/15/21 (six slices, FP64 s*m*2^e, e in [-20,20])"),
            "M": n, "N": n, "K": n, "calls_per_step": len(VARIANTS),
            "fp64_split_scope": args.scope,
        },
        "per_variant": per_variant,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
        "accuracy_uniform": accuracy,
        "mfma_frac_below_target": below_target,
        "inputs_sha256": sha,
        "domain_status": status,
        "context_peaks_tflops": {"bf16_mfma": PEAK_BF16_TFLOPS, "fp32_matrix": PEAK_FP32_MATRIX,
                                 "fp64_matrix": PEAK_FP64_MATRIX},
        "context_native_gemm": native,
        "context_other_depths": depths,
        "context_paper_8192": PAPER_CONTEXT_8192 if n == 8192 else None,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
