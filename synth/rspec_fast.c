/* Fast host implementation of the weight recipe in synth/rspec.py (same
 * definition, OpenMP over elements).  Input synthesis only. */
#include <stdint.h>

static inline uint64_t sm64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

void rspec_fill(uint64_t seed, uint64_t tid, uint64_t start, int64_t count, float *out) {
    const uint64_t key = sm64(seed ^ sm64(tid));
    union { uint32_t u; float f; } sc;
    sc.u = 0x310DE3BDu;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < count; ++t) {
        const uint64_t i = start + (uint64_t)t;
        const uint64_t r1 = sm64(key + 2 * i), r2 = sm64(key + 2 * i + 1);
        const uint64_t s = (r1 >> 40) + ((r1 >> 16) & 0xFFFFFF) + (r2 >> 40) + ((r2 >> 16) & 0xFFFFFF);
        const int32_t c = (int32_t)((int64_t)s - (1ll << 25));
        volatile float fc = (float)c;     /* round to nearest even, then one multiply */
        out[t] = fc * sc.f;
    }
}
