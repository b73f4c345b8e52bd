"""Seeded synthetic operands for the emulated-GEMM workloads.

This module is shared by the tests, the benchmark and the CPU oracle's callers.
It holds no arithmetic of the emulation method itself: it only turns a seed and
an element index into a reproducible random number and maps those numbers onto
the value distributions the paper and the workload list call for.

Generator: a counter-based SplitMix64.  Element ``i`` of stream ``seed`` is
``mix64(seed * 2**32 + i + 1)`` where ``mix64`` is SplitMix64's output function
applied to ``state = counter * 0x9E3779B97F4A7C15`` (the golden-ratio Weyl step
of the published generator).  No library distribution routine is used, so the
streams are stable across numpy versions.

Distributions (all computed in FP64; FP32 operands are one RNE cast of that):

* ``uniform``  : ``u = (x >> 11) * 2**-53`` in [0, 1);  value ``2u - 1`` in [-1, 1).
  Matches the paper's accuracy workload (uniform random entries in [-1, 1]).
* ``normal``   : Box-Muller with ``u1 = ((x0 >> 11) + 1) * 2**-53`` in (0, 1] and
  ``u2 = (x1 >> 11) * 2**-53``, value ``sqrt(-2 ln u1) * cos(2 pi u2)``.
* ``wide``     : ``s * m * 2**e`` with ``s`` = +-1 from bit 0 of ``x0``, ``e`` a
  uniform integer in [-20, 20] from the high 32 bits of ``x0`` (multiply-shift),
  and ``m = 1 + (x1 >> 12) * 2**-52`` in [1, 2).  This is the wide-dynamic-range
  class (scaled / log-uniform entries that stay inside the BF16 exponent range).
* ``normal_scaled_rows`` : ``normal`` with ceil(1 %) of the rows multiplied by
  2**16; the rows are the first entries of a seeded Fisher-Yates permutation.

Seeds: operand A of workload ``cfg`` uses ``1000*cfg + 1`` and B ``1000*cfg + 2``.

The bulk loops run in ``gen.c`` (built on first use with gcc into ``_gen.so``,
or by ``build()``); ``stream`` and ``element`` are also written out in plain
Python for checking it.
"""
from __future__ import annotations

import ctypes
import hashlib
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "_gen.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile gen.c into _gen.so (gcc, OpenMP, no FP contraction)."""
    src = os.path.join(_HERE, "gen.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                        "-shared", src, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _SO)
    return _SO


def _gen():
    global _lib
    if _lib is None:
        L = ctypes.CDLL(build())
        u64, i64, p, d, ci = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_double,
                              ctypes.c_int)
        L.sg_stream.argtypes = [u64, i64, i64, p]
        L.sg_uniform.argtypes = [u64, i64, d, d, p]
        L.sg_normal.argtypes = [u64, i64, p]
        L.sg_wide.argtypes = [u64, i64, ci, ci, p]
        for f in (L.sg_stream, L.sg_uniform, L.sg_normal, L.sg_wide):
            f.restype = None
        _lib = L
    return _lib


def _u64(seed: int) -> int:
    return int(seed) % (1 << 64)


def stream(seed: int, n: int, offset: int = 0) -> np.ndarray:
    """Elements ``offset .. offset+n-1`` of counter-based stream ``seed`` (uint64)."""
    out = np.empty(n, dtype=np.uint64)
    if n:
        _gen().sg_stream(_u64(seed), n, int(offset), out.ctypes.data)
    return out


def element(seed: int, i: int) -> int:
    """Element ``i`` of stream ``seed`` in plain Python integers (the definition)."""
    mask = (1 << 64) - 1
    z = ((((int(seed) << 32) + i + 1) & mask) * 0x9E3779B97F4A7C15) & mask
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & mask
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & mask
    return z ^ (z >> 31)


def uniform(seed: int, shape, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float64)
    if n:
        _gen().sg_uniform(_u64(seed), n, float(lo), float(hi), out.ctypes.data)
    return out.reshape(shape)


def normal(seed: int, shape) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float64)
    if n:
        _gen().sg_normal(_u64(seed), n, out.ctypes.data)
    return out.reshape(shape)


def wide(seed: int, shape, emin: int = -20, emax: int = 20) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float64)
    if n:
        _gen().sg_wide(_u64(seed), n, int(emin), int(emax), out.ctypes.data)
    return out.reshape(shape)


def value(dist: str, seed: int, i: int) -> float:
    """Element ``i`` of a distribution, in plain Python (checks the bulk loops)."""
    if dist == "uniform":
        return -1.0 + 2.0 * ((element(seed, i) >> 11) * 2.0 ** -53)
    x0, x1 = element(seed, 2 * i), element(seed, 2 * i + 1)
    if dist == "normal":
        u1 = ((x0 >> 11) + 1.0) * 2.0 ** -53
        u2 = (x1 >> 11) * 2.0 ** -53
        return math.sqrt(-2.0 * math.log(u1)) * math.cos(2.0 * math.pi * u2)
    if dist == "wide":
        s = -1.0 if x0 & 1 else 1.0
        e = (((x0 >> 32) * 41) >> 32) - 20
        return math.ldexp(s * (1.0 + (x1 >> 12) * 2.0 ** -52), e)
    raise ValueError(dist)


def permutation(seed: int, n: int) -> np.ndarray:
    """Seeded Fisher-Yates shuffle of 0..n-1 (Durstenfeld's in-place form)."""
    p = np.arange(n, dtype=np.int64)
    if n < 2:
        return p
    x = stream(seed, n - 1)
    for t, i in enumerate(range(n - 1, 0, -1)):
        j = int((int(x[t]) >> 32) * (i + 1) >> 32)
        p[i], p[j] = p[j], p[i]
    return p


def normal_scaled_rows(seed: int, shape, frac: float = 0.01, scale_exp: int = 16) -> np.ndarray:
    a = normal(seed, shape)
    rows = shape[0]
    k = int(np.ceil(frac * rows))
    pick = permutation(seed + 500, rows)[:k]
    a[pick, :] *= 2.0 ** scale_exp
    return a


def make(dist: str, seed: int, shape, dtype) -> np.ndarray:
    """Operand of the given distribution; FP32 operands are RNE-cast from FP64."""
    fn = {"uniform": uniform, "normal": normal, "wide": wide,
          "normal_scaled_rows": normal_scaled_rows}[dist]
    return np.ascontiguousarray(fn(seed, tuple(shape)).astype(dtype))


def seeds(cfg: int):
    return 1000 * cfg + 1, 1000 * cfg + 2


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


# The five workload families (shapes, value classes, product counts).
WORKLOADS = {
    1: dict(kind="sgemm", shapes=[(256, 256, 256)], dist="uniform"),
    2: dict(kind="sgemm", shapes=[(n, n, n) for n in (1024, 2048, 4096, 8192)], dist="normal"),
    3: dict(kind="dgemm", shapes=[(4096, 4096, 4096)], dist="uniform", nprod=(6, 10, 15, 21)),
    4: dict(kind="dgemm", shapes=[(8192, 8192, 8192), (16384, 16384, 16384)], dist="wide",
            nprod=(6, 21)),
    5: dict(kind="both", shapes=[(16384, 16384, 512), (1024, 1024, 65536)],
            dist="normal_scaled_rows", nprod=(10,)),
}
