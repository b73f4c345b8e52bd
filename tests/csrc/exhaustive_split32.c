/* Exhaustive check of the oracle's FP32 split over all 2^32 binary32 bit
   patterns (test helper, linked against the oracle library).

   For every finite a it checks, independently of the oracle's own rounding
   code:
     - A_0 equals round-to-nearest-even to BF16 written as the integer form
       (u + 0x7FFF + lsb) >> 16 on the bit pattern u;
     - whether a == A_0 + A_1 + A_2 exactly (the three BF16 values summed in
       binary64, which is exact for three 8-bit significands);
     - whether every component is a normal BF16 value or zero.
   It reports counts; the caller asserts that every a inside
   2^-103 <= |a| < (2 - 2^-8) 2^127 (and a = +-0) splits exactly into normal
   or zero components, as Sterbenz's lemma predicts (Sec. 4.2). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

extern unsigned orc_split_f32(int64_t R, int64_t C, const float *X, int64_t ldx, uint16_t *comps);

static float f_of(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static double bf(uint16_t h) { return (double)f_of((uint32_t)h << 16); }
static int normal_or_zero(uint16_t h) {
    int ex = (h >> 7) & 0xFF, fr = h & 0x7F;
    if (ex == 0xFF) return 0;
    if (ex == 0 && fr != 0) return 0;
    return 1;
}

int main(int argc, char **argv) {
    uint64_t lo = 0, hi = 1ull << 32;
    if (argc >= 3) { lo = strtoull(argv[1], 0, 0); hi = strtoull(argv[2], 0, 0); }
    const int64_t R = 4096, C = 1024, CH = R * C;
    float *X = (float *)malloc(CH * sizeof(float));
    uint16_t *comps = (uint16_t *)malloc(3 * CH * sizeof(uint16_t));
    unsigned long long n_finite = 0, n_in = 0, bad_in = 0, rne_bad = 0, fail_out = 0, fail_low = 0,
                       fail_high = 0;
    for (uint64_t base = lo; base < hi; base += CH) {
        int64_t n = (hi - base) < (uint64_t)CH ? (int64_t)(hi - base) : CH;
        for (int64_t i = 0; i < CH; ++i) X[i] = f_of((uint32_t)(base + (uint64_t)(i < n ? i : 0)));
        orc_split_f32(R, C, X, C, comps);
#pragma omp parallel for reduction(+ : n_finite, n_in, bad_in, rne_bad, fail_out, fail_low, fail_high)
        for (int64_t i = 0; i < n; ++i) {
            uint32_t u = (uint32_t)(base + (uint64_t)i);
            float a = f_of(u);
            if (!isfinite(a)) continue;
            n_finite++;
            uint16_t c0 = comps[i], c1 = comps[CH + i], c2 = comps[2 * CH + i];
            uint16_t ref0 = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
            if (c0 != ref0) rne_bad++;
            int ok = normal_or_zero(c0) && normal_or_zero(c1) && normal_or_zero(c2) &&
                     (bf(c0) + bf(c1) + bf(c2) == (double)a);
            double aa = fabs((double)a);
            int in = (a == 0.0f) || (aa >= ldexp(1.0, -103) && aa < ldexp(2.0 - ldexp(1.0, -8), 127));
            if (in) { n_in++; if (!ok) bad_in++; }
            else if (!ok) { fail_out++; if (aa < 1.0) fail_low++; else fail_high++; }
        }
    }
    printf("%llu %llu %llu %llu %llu %llu %llu\n", n_finite, n_in, bad_in, rne_bad, fail_out,
           fail_low, fail_high);
    free(X);
    free(comps);
    return 0;
}
