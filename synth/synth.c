/*
 * Seeded synthetic inputs for the attention workloads.
 *
 * This file holds random-number generation and storage conversion only; it
 * contains no part of the attention computation.  Both the fp64 oracle tests
 * and the GPU tests draw their Q, K and V from here, so the two sides see the
 * same bytes.
 *
 * Generator: counter-based SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  Output k of a stream with
 * seed s is mix64(s + (k + 1) * 0x9E3779B97F4A7C15), which equals the k-th value
 * of the sequential generator started at state s.
 *   mix64(z): z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9;
 *             z = (z ^ (z >> 27)) * 0x94D049BB133111EB;
 *             return z ^ (z >> 31);
 * Uniform: u = (x >> 11) * 2^-53, in [0, 1).
 * Normal: Box-Muller on the pair (u1, u2) = (output 2p, output 2p + 1):
 *   r = sqrt(-2 ln(1 - u1)), theta = 2 pi u2,
 *   element 2p = r cos(theta), element 2p + 1 = r sin(theta).
 * The fp64 normal is multiplied by sigma, rounded to fp32 (C cast,
 * round-to-nearest-even), and for bf16 storage rounded again to bf16 with
 * round-to-nearest-even on the fp32 bit pattern.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static const uint64_t GOLDEN = 0x9E3779B97F4A7C15ULL;

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t synth_splitmix64(uint64_t seed, uint64_t k) {
    return mix64(seed + (k + 1) * GOLDEN);
}

static inline double uniform01(uint64_t seed, uint64_t k) {
    return (double)(synth_splitmix64(seed, k) >> 11) * 0x1.0p-53;
}

/* Element i of the N(0, sigma^2) stream, in fp64. */
static inline double normal_at(uint64_t seed, int64_t i, double sigma) {
    const double two_pi = 6.283185307179586476925286766559;
    uint64_t p = (uint64_t)(i >> 1);
    double u1 = uniform01(seed, 2 * p);
    double u2 = uniform01(seed, 2 * p + 1);
    double r = sqrt(-2.0 * log(1.0 - u1));
    double th = two_pi * u2;
    double z = (i & 1) ? r * sin(th) : r * cos(th);
    return z * sigma;
}

/* fp32 -> bf16 bits, round to nearest even (inputs here are always finite). */
static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

void synth_normal_f64(uint64_t seed, int64_t n, double sigma, double* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = normal_at(seed, i, sigma);
}

void synth_normal_f32(uint64_t seed, int64_t n, double sigma, float* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)normal_at(seed, i, sigma);
}

void synth_normal_bf16(uint64_t seed, int64_t n, double sigma, uint16_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne((float)normal_at(seed, i, sigma));
}

/* Storage conversion used when a test builds inputs from fp32 values. */
void synth_f32_to_bf16(const float* in, int64_t n, uint16_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne(in[i]);
}
