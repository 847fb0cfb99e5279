/*
 * Seeded synthetic inputs for the single-stage forward: Gaussian samples from a
 * counter-based generator, written as bf16 bits (weights, norm gains) or fp32
 * (hidden states).  This file holds random-number generation only; it computes
 * nothing of the decoder layer.  It serves both the oracle and the HIP path, so
 * both consume identical bits.
 *
 * Generator (all arithmetic is exact integer or IEEE double):
 *   SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
 *   generators", OOPSLA 2014): the k-th draw (k = 0, 1, ...) of stream `seed` is
 *       mix64(seed + (k + 1) * 0x9E3779B97F4A7C15)  (mod 2^64)
 *   with mix64 the variant-13 finaliser below.
 *   Box-Muller (Box & Muller 1958): element i of a stream uses draws 2*(i/2) and
 *   2*(i/2)+1:  u1 = ((d0 >> 11) + 0.5) * 2^-53  (in (0,1)),  u2 = (d1 >> 11) * 2^-53,
 *   r = sqrt(-2 ln u1),  z = r cos(2 pi u2) for even i, r sin(2 pi u2) for odd i.
 *   value = mean + std * z, evaluated in double, rounded to float (nearest even),
 *   then for bf16 outputs rounded float -> bf16 (nearest even).
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC gen.c -o _libsynth.so -lm
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t seed, uint64_t k) {
    return mix64(seed + (k + 1ULL) * 0x9E3779B97F4A7C15ULL);
}

/* Both Box-Muller outputs of pair p: z[0] for element 2p, z[1] for element 2p+1. */
static inline void gauss_pair(uint64_t seed, uint64_t p, double z[2]) {
    const uint64_t d0 = draw(seed, 2 * p), d1 = draw(seed, 2 * p + 1);
    const double u1 = ((double)(d0 >> 11) + 0.5) * 0x1.0p-53;
    const double u2 = (double)(d1 >> 11) * 0x1.0p-53;
    const double r = sqrt(-2.0 * log(u1));
    const double a = 6.283185307179586476925286766559 * u2;
    double sn, cs;
    sincos(a, &sn, &cs);
    z[0] = r * cs;
    z[1] = r * sn;
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* Calls emit(j, z) for every j in [0, n) with z the Gaussian of element offset + j. */
#define SYNTH_FILL(EMIT)                                                            \
    do {                                                                            \
        const uint64_t first = offset, last = offset + (uint64_t)n; /* [first,last) */ \
        const int64_t p0 = (int64_t)(first >> 1), p1 = (int64_t)((last + 1) >> 1);   \
        _Pragma("omp parallel for schedule(static)")                                \
        for (int64_t p = p0; p < p1; ++p) {                                          \
            double z[2];                                                            \
            gauss_pair(seed, (uint64_t)p, z);                                       \
            for (int e = 0; e < 2; ++e) {                                           \
                const uint64_t c = 2 * (uint64_t)p + (uint64_t)e;                   \
                if (c < first || c >= last) continue;                               \
                const int64_t j = (int64_t)(c - first);                             \
                EMIT;                                                               \
            }                                                                       \
        }                                                                           \
    } while (0)

/* out[j] = bf16(float(mean + std * z_{offset+j})), j in [0, n). */
void synth_normal_bf16(uint64_t seed, uint64_t offset, int64_t n, double mean, double std, uint16_t *out) {
    SYNTH_FILL(out[j] = f32_to_bf16_rne((float)(mean + std * z[e])));
}

/* out[j] = float(mean + std * z_{offset+j}), j in [0, n). */
void synth_normal_f32(uint64_t seed, uint64_t offset, int64_t n, double mean, double std, float *out) {
    SYNTH_FILL(out[j] = (float)(mean + std * z[e]));
}

/* Raw 64-bit draws, for checking the generator against its definition. */
void synth_draws(uint64_t seed, uint64_t offset, int64_t n, uint64_t *out) {
    for (int64_t j = 0; j < n; ++j) out[j] = draw(seed, offset + (uint64_t)j);
}
