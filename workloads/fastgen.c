/* Compiled twin of the normal generator in gen.py (same definitions):
 * counter-based SplitMix64 (Steele, Lea & Flood 2014) and the Box-Muller
 * transform in fp64, cast to fp32.  Draw i of stream `key` is
 * mix64(key + (i + 1) * GAMMA); normal pair j uses draws 2j and 2j + 1.
 * Each output depends only on its index, so the thread count does not change
 * the result.  Input generation only: nothing of the method is computed here. */
#include <math.h>
#include <stdint.h>

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline double u53(uint64_t key, uint64_t i) {
    return (double)(mix64(key + (i + 1) * 0x9E3779B97F4A7C15ULL) >> 11) * 0x1.0p-53;
}

void wl_normal_f32(uint64_t key, int64_t n, double sigma, float *out) {
    const int64_t npairs = (n + 1) / 2;
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < npairs; ++j) {
        const double u1 = u53(key, (uint64_t)(2 * j));
        const double u2 = u53(key, (uint64_t)(2 * j + 1));
        const double r = sqrt(-2.0 * log1p(-u1));
        const double th = two_pi * u2;
        out[2 * j] = (float)(sigma * (r * cos(th)));
        if (2 * j + 1 < n) out[2 * j + 1] = (float)(sigma * (r * sin(th)));
    }
}
