/* Seeded synthetic input generator shared by the HIP path and the CPU oracle.
 *
 * It draws numbers and rounds them to the storage type; it contains none of
 * the operators' arithmetic.  Counter-based SplitMix64 (Steele, Lea and
 * Flood, OOPSLA 2014): element i of tensor tid under seed is
 *   mix64(key(seed, tid) + (i + 1) * GAMMA).
 * Uniform doubles use the top 53 bits; normals use Box-Muller on counters
 * (2i, 2i+1) with u1 = 1 - uniform in (0, 1].  fp64 -> fp32 is round to
 * nearest even; fp32 -> bf16 is round to nearest even on the bit pattern.
 * Every element is independent, so the result does not depend on the
 * number of OpenMP threads.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t tid) {
    return mix64(seed * 0x100000001B3ULL + tid * 0x9E3779B1ULL);
}

static inline double u53(uint64_t h) { return (double)(h >> 11) * (1.0 / 9007199254740992.0); }

static inline uint16_t f32_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

static inline double normal_at(uint64_t key, int64_t i) {
    double u1 = 1.0 - u53(mix64(key + (uint64_t)(2 * i + 1) * GAMMA));
    double u2 = u53(mix64(key + (uint64_t)(2 * i + 2) * GAMMA));
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}

void synth_u64(uint64_t seed, uint64_t tid, int64_t start, int64_t n, uint64_t *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = mix64(key + (uint64_t)(start + i + 1) * GAMMA);
}

void synth_uniform_f32(uint64_t seed, uint64_t tid, int64_t n, double lo, double hi, float *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)(lo + (hi - lo) * u53(mix64(key + (uint64_t)(i + 1) * GAMMA)));
}

void synth_normal_f32(uint64_t seed, uint64_t tid, int64_t n, double sigma, float *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)(sigma * normal_at(key, i));
}

void synth_normal_bf16(uint64_t seed, uint64_t tid, int64_t n, double sigma, uint16_t *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = f32_bf16((float)(sigma * normal_at(key, i)));
}

/* Integers uniform in [-a, a], stored as bf16 (exact for |v| <= 256). */
void synth_int_bf16(uint64_t seed, uint64_t tid, int64_t n, int32_t a, uint16_t *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double u = u53(mix64(key + (uint64_t)(i + 1) * GAMMA));
        out[i] = f32_bf16((float)(floor(u * (2.0 * a + 1.0)) - a));
    }
}

/* Integers uniform in [-a, a], stored as fp32. */
void synth_int_f32(uint64_t seed, uint64_t tid, int64_t n, int32_t a, float *out) {
    uint64_t key = stream_key(seed, tid);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double u = u53(mix64(key + (uint64_t)(i + 1) * GAMMA));
        out[i] = (float)(floor(u * (2.0 * a + 1.0)) - a);
    }
}
