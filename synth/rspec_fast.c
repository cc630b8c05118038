/* Fast host implementation of the weight recipe in synth/rspec.py (same
 * definition, OpenMP over elements).  Input synthesis only. */
#include <stdint.h>
#include <string.h>

static inline uint64_t sm64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* element i of the tensor keyed by `key`: float(int(S - 2^25)) * C, both
 * operations rounding to nearest even (compiled without FP contraction) */
static inline float rspec_value(uint64_t key, uint64_t i) {
    const uint64_t r1 = sm64(key + 2 * i), r2 = sm64(key + 2 * i + 1);
    const uint64_t s = (r1 >> 40) + ((r1 >> 16) & 0xFFFFFF) + (r2 >> 40) + ((r2 >> 16) & 0xFFFFFF);
    const int32_t c = (int32_t)((int64_t)s - (1ll << 25));
    uint32_t cu = 0x310DE3BDu;
    float scale;
    memcpy(&scale, &cu, 4);
    return (float)c * scale;
}

static inline float round_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u = ((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16) << 16;
    memcpy(&f, &u, 4);
    return f;
}

/* round_bf16 != 0: round each value to the nearest bf16 (ties to even) */
void rspec_fill(uint64_t seed, uint64_t tid, uint64_t start, int64_t count, float *out, int rb) {
    const uint64_t key = sm64(seed ^ sm64(tid));
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < count; ++t) {
        const float w = rspec_value(key, start + (uint64_t)t);
        out[t] = rb ? round_bf16(w) : w;
    }
}

/* the same values written as float64 */
void rspec_fill64(uint64_t seed, uint64_t tid, uint64_t start, int64_t count, double *out, int rb) {
    const uint64_t key = sm64(seed ^ sm64(tid));
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < count; ++t) {
        const float w = rspec_value(key, start + (uint64_t)t);
        out[t] = (double)(rb ? round_bf16(w) : w);
    }
}
