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
"""
from __future__ import annotations

import hashlib

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_CHUNK = 1 << 22


def _mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function (Steele, Lea, Flood 2014), on uint64 arrays."""
    z = z.copy()
    z ^= z >> np.uint64(30)
    z *= _M1
    z ^= z >> np.uint64(27)
    z *= _M2
    z ^= z >> np.uint64(31)
    return z


def stream(seed: int, n: int, offset: int = 0) -> np.ndarray:
    """Elements ``offset .. offset+n-1`` of counter-based stream ``seed`` (uint64)."""
    out = np.empty(n, dtype=np.uint64)
    base = (int(seed) << 32) + int(offset) + 1
    with np.errstate(over="ignore"):
        for s in range(0, n, _CHUNK):
            e = min(n, s + _CHUNK)
            ctr = (np.arange(s, e, dtype=np.uint64) + np.uint64(base % (1 << 64)))
            out[s:e] = _mix64(ctr * _GAMMA)
    return out


def _unit53(x: np.ndarray) -> np.ndarray:
    return (x >> np.uint64(11)).astype(np.float64) * 2.0 ** -53


def uniform(seed: int, shape, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    n = int(np.prod(shape))
    u = _unit53(stream(seed, n))
    return (lo + (hi - lo) * u).reshape(shape)


def normal(seed: int, shape) -> np.ndarray:
    n = int(np.prod(shape))
    x = stream(seed, 2 * n)
    u1 = ((x[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * 2.0 ** -53
    u2 = _unit53(x[1::2])
    return (np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)).reshape(shape)


def wide(seed: int, shape, emin: int = -20, emax: int = 20) -> np.ndarray:
    n = int(np.prod(shape))
    x = stream(seed, 2 * n)
    x0, x1 = x[0::2], x[1::2]
    sign = np.where((x0 & np.uint64(1)) == 0, 1.0, -1.0)
    span = np.uint64(emax - emin + 1)
    with np.errstate(over="ignore"):
        e = ((x0 >> np.uint64(32)) * span) >> np.uint64(32)
    e = e.astype(np.int64) + emin
    m = 1.0 + (x1 >> np.uint64(12)).astype(np.float64) * 2.0 ** -52
    return np.ldexp(sign * m, e.astype(np.int32)).reshape(shape)


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
