/* Counter-based normal sampling for the synthetic workload generator.
 *
 * Element i of stream s under seed `seed`:
 *   key  = mix(seed * 2^32 + s + GAMMA)
 *   u64  = mix(key + (i + 1) * GAMMA)          (mod 2^64)
 * where mix() is the SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014).
 * Uniforms in (0, 1] are ((u64 >> 11) + 1) * 2^-53; normal i is the cosine
 * branch of Box-Muller on uniforms 2i and 2i+1.  Values are scaled by `std`,
 * rounded to float32 (RNE) and, for the bf16 entry point, then to bf16 (RNE
 * on the float32 bit pattern).
 *
 * Every element depends only on its own counter, so the OpenMP split does not
 * change any value.  This file holds no verification arithmetic.
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

static inline uint64_t stream_key(uint64_t seed, uint32_t stream) {
    return mix64(((seed & 0xFFFFFFFFULL) << 32) + (uint64_t)stream + GAMMA);
}

static inline double unit(uint64_t key, uint64_t i) {
    uint64_t u = mix64(key + (i + 1) * GAMMA);
    return ((double)(u >> 11) + 1.0) * 0x1.0p-53;
}

static inline double normal_at(uint64_t key, uint64_t i) {
    double u1 = unit(key, 2 * i), u2 = unit(key, 2 * i + 1);
    return sqrt(-2.0 * log(u1)) * cos((2.0 * M_PI) * u2);
}

static inline uint16_t f32_to_bf16(float f) {
    uint32_t b;
    memcpy(&b, &f, 4);
    b = b + 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

void synth_normal_f32(uint64_t seed, uint32_t stream, uint64_t start, int64_t count,
                      double std, float* out) {
    uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = (float)(normal_at(key, start + (uint64_t)i) * std);
}

void synth_normal_bf16(uint64_t seed, uint32_t stream, uint64_t start, int64_t count,
                       double std, uint16_t* out) {
    uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = f32_to_bf16((float)(normal_at(key, start + (uint64_t)i) * std));
}
