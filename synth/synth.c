/*
 * Seeded synthetic inputs for the DVI decode step: weights, prompts and
 * replay-buffer contents.  This file holds no arithmetic of the method
 * itself; it only draws numbers.  Both the CPU oracle and the GPU path take
 * their inputs from here, so the two see bit-identical arrays.
 *
 * Generator: counter-based.  Every value is a pure function of
 * (seed, stream id, element index), so the result does not depend on the
 * number of threads or on which slice of an array is generated.
 *
 *   key(seed, stream) = mix64(mix64(seed) ^ (stream * GOLDEN))
 *   bits(key, c)      = mix64(key + (c + 1) * GOLDEN)
 *
 * mix64 is the SplitMix64 output finaliser (Steele, Lea & Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014; constants of
 * Stafford's "variant 13").  A uniform in (0,1) is ((bits >> 11) + 0.5)/2^53.
 * Normals come from the Box-Muller transform (Box & Muller, 1958) on the
 * uniform pair (2j, 2j+1): element 2j takes the cosine branch, 2j+1 the sine
 * branch.  The double result is scaled by std, rounded to float (RNE), and
 * for bf16 arrays rounded again to bf16 (RNE on the float bit pattern).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
    return mix64(mix64(seed) ^ (stream * GOLDEN));
}

static inline uint64_t bits_at(uint64_t key, uint64_t c) {
    return mix64(key + (c + 1) * GOLDEN);
}

static inline double unif_at(uint64_t key, uint64_t c) {
    return ((double)(bits_at(key, c) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40); /* NaN */
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

/* Both Box-Muller branches of pair j: elements 2j (cosine) and 2j+1 (sine). */
static inline void normal_pair(uint64_t key, uint64_t j, double *z0, double *z1) {
    double u1 = unif_at(key, 2 * j);
    double u2 = unif_at(key, 2 * j + 1);
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925 * u2;
    *z0 = rad * cos(ang);
    *z1 = rad * sin(ang);
}

/* out[i] = (float)(std * N(0,1)_i) for i in [0, n) */
void synth_normal_f32(uint64_t seed, uint64_t stream, double std, int64_t n, float *out) {
    uint64_t key = stream_key(seed, stream);
    int64_t np_ = (n + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < np_; ++j) {
        double z0, z1;
        normal_pair(key, (uint64_t)j, &z0, &z1);
        out[2 * j] = (float)(std * z0);
        if (2 * j + 1 < n) out[2 * j + 1] = (float)(std * z1);
    }
}

/* out[i] = bf16 bits of (float)(std * N(0,1)_i) */
void synth_normal_bf16(uint64_t seed, uint64_t stream, double std, int64_t n, uint16_t *out) {
    uint64_t key = stream_key(seed, stream);
    int64_t np_ = (n + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < np_; ++j) {
        double z0, z1;
        normal_pair(key, (uint64_t)j, &z0, &z1);
        out[2 * j] = f32_to_bf16_rne((float)(std * z0));
        if (2 * j + 1 < n) out[2 * j + 1] = f32_to_bf16_rne((float)(std * z1));
    }
}

/* out[i] uniform integer in [0, hi): floor(u * hi) */
void synth_uniform_int(uint64_t seed, uint64_t stream, int32_t hi, int64_t n, int32_t *out) {
    uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t v = (int64_t)(unif_at(key, (uint64_t)i) * (double)hi);
        if (v >= hi) v = hi - 1;
        out[i] = (int32_t)v;
    }
}

/* out[i] uniform double in (0, 1) */
void synth_uniform_f64(uint64_t seed, uint64_t stream, int64_t n, double *out) {
    uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = unif_at(key, (uint64_t)i);
}

/* raw 64-bit outputs, exposed so tests can check the generator itself */
void synth_bits(uint64_t seed, uint64_t stream, int64_t n, uint64_t *out) {
    uint64_t key = stream_key(seed, stream);
    for (int64_t i = 0; i < n; ++i) out[i] = bits_at(key, (uint64_t)i);
}

uint64_t synth_mix64(uint64_t z) { return mix64(z); }
