/*
 * Bulk form of the seeded operand generator (see __init__.py for the
 * definitions).  Counter-based, so every element is computed independently and
 * the loops run in parallel; compiled with -ffp-contract=off so that every
 * floating-point expression rounds exactly as written.
 */
#include <math.h>
#include <stdint.h>

static inline uint64_t mix64(uint64_t z) {
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

/* element i of stream seed */
static inline uint64_t draw(uint64_t seed, uint64_t i) {
    return mix64(((seed << 32) + i + 1) * 0x9E3779B97F4A7C15ull);
}

void sg_stream(uint64_t seed, int64_t n, int64_t offset, uint64_t *out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = draw(seed, (uint64_t)(offset + i));
}

void sg_uniform(uint64_t seed, int64_t n, double lo, double hi, double *out) {
    const double w = hi - lo;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const double u = (double)(draw(seed, (uint64_t)i) >> 11) * 0x1p-53;
        out[i] = lo + w * u;
    }
}

void sg_normal(uint64_t seed, int64_t n, double *out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const uint64_t x0 = draw(seed, 2 * (uint64_t)i), x1 = draw(seed, 2 * (uint64_t)i + 1);
        const double u1 = ((double)(x0 >> 11) + 1.0) * 0x1p-53;
        const double u2 = (double)(x1 >> 11) * 0x1p-53;
        out[i] = sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
    }
}

void sg_wide(uint64_t seed, int64_t n, int emin, int emax, double *out) {
    const uint64_t span = (uint64_t)(emax - emin + 1);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const uint64_t x0 = draw(seed, 2 * (uint64_t)i), x1 = draw(seed, 2 * (uint64_t)i + 1);
        const double s = (x0 & 1) ? -1.0 : 1.0;
        const int e = (int)(((x0 >> 32) * span) >> 32) + emin;
        const double m = 1.0 + (double)(x1 >> 12) * 0x1p-52;
        out[i] = ldexp(s * m, e);
    }
}
